// MS-LN / MS-RMSNorm kernels for gfx950 (Sec. 5.2 Alg. 1; Appendix G Alg. 2, Alg. 3).
//
// Forward, per row x of width p: sigma = sqrt(p^-1 |H x|^2 + eps), z = H x / sigma,
// rstd = 1 / sigma, where H x = x - mean(x) (LN) or x (RMS). Backward from the saved
// output alone: dx = rstd * (H dz - z * p^-1 z^T dz).
//
// Fast path: one wave per row, the row held in registers (VPL 16-byte vectors per
// lane, lane l holding vectors l, l + 64, ...), so each tensor is read from HBM once
// and every statistic is a register pass plus a wave reduction. Rows that are not
// 16-byte aligned, or wider than the register tile, use a block-per-row path that
// re-reads the row for each pass.
//
// Numerics: LN accumulates x - x0 (x0 = the row's first element) so that rows
// with a large common offset do not lose the deviations to rounding; the centred
// values are (x - x0) - mean(x - x0), never x - mean(x) with mean(x) rounded.
// Variances are two-pass over the register-resident row.
#include "lmbp_device.hpp"
#include "lmbp_launch.hpp"

namespace lmbp {

template <class IO>
__device__ inline float first_elem(const u32x4& v) {
  float f[IO::kPerVec];
  IO::unpack(v, f);
  return f[0];
}

template <class IO, bool LN, int VPL>
__global__ __launch_bounds__(256) void norm_fwd_vec(const void* x, void* z, float* __restrict__ rstd,
                                                    int64_t rows, int cols, float eps) {
  constexpr int E = IO::kPerVec;
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t row = int64_t(blockIdx.x) * (blockDim.x / kWave) + (threadIdx.x / kWave);
  if (row >= rows) return;
  const int nv = cols / E;
  const int64_t vbase = row * nv;

  u32x4 v[VPL];
#pragma unroll
  for (int j = 0; j < VPL; ++j) {
    const int idx = j * kWave + lane;
    v[j] = (idx < nv) ? ldg16(x, vbase + idx) : u32x4{0u, 0u, 0u, 0u};
  }

  float pivot = 0.0f, mean_d = 0.0f;
  if constexpr (LN) {
    pivot = __builtin_bit_cast(float, __builtin_amdgcn_readfirstlane(
                                          __builtin_bit_cast(int, first_elem<IO>(v[0]))));
    float s1 = 0.0f;
#pragma unroll
    for (int j = 0; j < VPL; ++j) {
      if (j * kWave + lane < nv) {
        float f[E];
        IO::unpack(v[j], f);
#pragma unroll
        for (int e = 0; e < E; ++e) s1 += f[e] - pivot;
      }
    }
    mean_d = wave_sum(s1) / float(cols);
  }

  float s2 = 0.0f;
#pragma unroll
  for (int j = 0; j < VPL; ++j) {
    if (j * kWave + lane < nv) {
      float f[E];
      IO::unpack(v[j], f);
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const float c = LN ? (f[e] - pivot) - mean_d : f[e];
        s2 = __builtin_fmaf(c, c, s2);
      }
    }
  }
  const float var = wave_sum(s2) / float(cols);
  const float rs = rsqrtf(var + eps);

#pragma unroll
  for (int j = 0; j < VPL; ++j) {
    const int idx = j * kWave + lane;
    if (idx < nv) {
      float f[E];
      IO::unpack(v[j], f);
#pragma unroll
      for (int e = 0; e < E; ++e) f[e] = (LN ? (f[e] - pivot) - mean_d : f[e]) * rs;
      stg16(z, vbase + idx, IO::pack(f));
    }
  }
  if (lane == 0) rstd[row] = rs;
}

template <class IO, bool LN, int VPL>
__global__ __launch_bounds__(256) void norm_bwd_vec(const void* dz, const void* z,
                                                    const float* __restrict__ rstd, void* dx,
                                                    int64_t rows, int cols) {
  constexpr int E = IO::kPerVec;
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t row = int64_t(blockIdx.x) * (blockDim.x / kWave) + (threadIdx.x / kWave);
  if (row >= rows) return;
  const int nv = cols / E;
  const int64_t vbase = row * nv;

  u32x4 vg[VPL], vz[VPL];
#pragma unroll
  for (int j = 0; j < VPL; ++j) {
    const int idx = j * kWave + lane;
    const bool ok = idx < nv;
    vg[j] = ok ? ldg16(dz, vbase + idx) : u32x4{0u, 0u, 0u, 0u};
    vz[j] = ok ? ldg16(z, vbase + idx) : u32x4{0u, 0u, 0u, 0u};
  }
  const float rs = rstd[row];

  // Zero padding contributes nothing to either sum.
  float s_g = 0.0f, s_zg = 0.0f;
#pragma unroll
  for (int j = 0; j < VPL; ++j) {
    float g[E], zz[E];
    IO::unpack(vg[j], g);
    IO::unpack(vz[j], zz);
#pragma unroll
    for (int e = 0; e < E; ++e) {
      if constexpr (LN) s_g += g[e];
      s_zg = __builtin_fmaf(zz[e], g[e], s_zg);
    }
  }
  const float a = LN ? wave_sum(s_g) / float(cols) : 0.0f;
  const float b = wave_sum(s_zg) / float(cols);

#pragma unroll
  for (int j = 0; j < VPL; ++j) {
    const int idx = j * kWave + lane;
    if (idx < nv) {
      float g[E], zz[E];
      IO::unpack(vg[j], g);
      IO::unpack(vz[j], zz);
#pragma unroll
      for (int e = 0; e < E; ++e) g[e] = rs * __builtin_fmaf(-zz[e], b, g[e] - a);
      stg16(dx, vbase + idx, IO::pack(g));
    }
  }
}

// Block per row, any alignment and width; each pass re-reads the row (from cache
// for rows that fit).
template <class IO, bool LN>
__global__ __launch_bounds__(256) void norm_fwd_any(const void* x, void* z, float* __restrict__ rstd,
                                                    int64_t rows, int64_t cols, float eps) {
  __shared__ float red[256 / kWave];
  const int64_t row = blockIdx.x;
  if (row >= rows) return;
  const int64_t base = row * cols;
  const int tid = threadIdx.x;

  float pivot = 0.0f, mean_d = 0.0f;
  if constexpr (LN) {
    pivot = IO::load1(x, base);
    float s1 = 0.0f;
    for (int64_t k = tid; k < cols; k += blockDim.x) s1 += IO::load1(x, base + k) - pivot;
    mean_d = block_sum(s1, red) / float(cols);
  }
  float s2 = 0.0f;
  for (int64_t k = tid; k < cols; k += blockDim.x) {
    const float f = IO::load1(x, base + k);
    const float c = LN ? (f - pivot) - mean_d : f;
    s2 = __builtin_fmaf(c, c, s2);
  }
  const float var = block_sum(s2, red) / float(cols);
  const float rs = rsqrtf(var + eps);
  for (int64_t k = tid; k < cols; k += blockDim.x) {
    const float f = IO::load1(x, base + k);
    IO::store1(z, base + k, (LN ? (f - pivot) - mean_d : f) * rs);
  }
  if (tid == 0) rstd[row] = rs;
}

template <class IO, bool LN>
__global__ __launch_bounds__(256) void norm_bwd_any(const void* dz, const void* z,
                                                    const float* __restrict__ rstd, void* dx,
                                                    int64_t rows, int64_t cols) {
  __shared__ float red[256 / kWave];
  const int64_t row = blockIdx.x;
  if (row >= rows) return;
  const int64_t base = row * cols;
  const int tid = threadIdx.x;

  float s_g = 0.0f, s_zg = 0.0f;
  for (int64_t k = tid; k < cols; k += blockDim.x) {
    const float g = IO::load1(dz, base + k);
    if constexpr (LN) s_g += g;
    s_zg = __builtin_fmaf(IO::load1(z, base + k), g, s_zg);
  }
  const float a = LN ? block_sum(s_g, red) / float(cols) : 0.0f;
  const float b = block_sum(s_zg, red) / float(cols);
  const float rs = rstd[row];
  for (int64_t k = tid; k < cols; k += blockDim.x) {
    const float g = IO::load1(dz, base + k);
    const float zz = IO::load1(z, base + k);
    IO::store1(dx, base + k, rs * __builtin_fmaf(-zz, b, g - a));
  }
}

// ------------------------------------------------------------------ launchers
namespace {
// Register tiles available to the fast path, in 16-byte vectors per lane.
constexpr int kVplChoices[] = {1, 2, 3, 4, 6, 8, 12, 16};
constexpr int kMaxVpl = 16;

template <class IO, bool LN, int VPL>
hipError_t fwd_vec(int64_t rows, int cols, float eps, const void* x, void* z, float* rstd,
                   hipStream_t s) {
  const int64_t blocks = (rows + 3) / 4;
  hipLaunchKernelGGL((norm_fwd_vec<IO, LN, VPL>), dim3(unsigned(blocks)), dim3(256), 0, s, x, z, rstd,
                     rows, cols, eps);
  return hipGetLastError();
}
template <class IO, bool LN, int VPL>
hipError_t bwd_vec(int64_t rows, int cols, const void* dz, const void* z, const float* rstd,
                   void* dx, hipStream_t s) {
  const int64_t blocks = (rows + 3) / 4;
  hipLaunchKernelGGL((norm_bwd_vec<IO, LN, VPL>), dim3(unsigned(blocks)), dim3(256), 0, s, dz, z, rstd,
                     dx, rows, cols);
  return hipGetLastError();
}

template <class IO>
int pick_vpl(int64_t cols) {
  const int64_t nv = cols / IO::kPerVec;
  for (int v : kVplChoices)
    if (int64_t(kWave) * v >= nv) return v;
  return 0;
}

template <class IO, bool LN>
hipError_t norm_fwd_t(int64_t rows, int64_t cols, float eps, const void* x, void* z, float* rstd,
                      bool vec_ok, hipStream_t s) {
  const int vpl = vec_ok ? pick_vpl<IO>(cols) : 0;
  if (vpl > 0 && (rows + 3) / 4 <= 0x7fffffff) {
    const int c = int(cols);
    switch (vpl) {
      case 1: return fwd_vec<IO, LN, 1>(rows, c, eps, x, z, rstd, s);
      case 2: return fwd_vec<IO, LN, 2>(rows, c, eps, x, z, rstd, s);
      case 3: return fwd_vec<IO, LN, 3>(rows, c, eps, x, z, rstd, s);
      case 4: return fwd_vec<IO, LN, 4>(rows, c, eps, x, z, rstd, s);
      case 6: return fwd_vec<IO, LN, 6>(rows, c, eps, x, z, rstd, s);
      case 8: return fwd_vec<IO, LN, 8>(rows, c, eps, x, z, rstd, s);
      case 12: return fwd_vec<IO, LN, 12>(rows, c, eps, x, z, rstd, s);
      default: return fwd_vec<IO, LN, kMaxVpl>(rows, c, eps, x, z, rstd, s);
    }
  }
  if (rows > 0x7fffffff) return hipErrorInvalidValue;
  hipLaunchKernelGGL((norm_fwd_any<IO, LN>), dim3(unsigned(rows)), dim3(256), 0, s, x, z, rstd, rows,
                     cols, eps);
  return hipGetLastError();
}

template <class IO, bool LN>
hipError_t norm_bwd_t(int64_t rows, int64_t cols, const void* dz, const void* z, const float* rstd,
                      void* dx, bool vec_ok, hipStream_t s) {
  const int vpl = vec_ok ? pick_vpl<IO>(cols) : 0;
  if (vpl > 0 && (rows + 3) / 4 <= 0x7fffffff) {
    const int c = int(cols);
    switch (vpl) {
      case 1: return bwd_vec<IO, LN, 1>(rows, c, dz, z, rstd, dx, s);
      case 2: return bwd_vec<IO, LN, 2>(rows, c, dz, z, rstd, dx, s);
      case 3: return bwd_vec<IO, LN, 3>(rows, c, dz, z, rstd, dx, s);
      case 4: return bwd_vec<IO, LN, 4>(rows, c, dz, z, rstd, dx, s);
      case 6: return bwd_vec<IO, LN, 6>(rows, c, dz, z, rstd, dx, s);
      case 8: return bwd_vec<IO, LN, 8>(rows, c, dz, z, rstd, dx, s);
      case 12: return bwd_vec<IO, LN, 12>(rows, c, dz, z, rstd, dx, s);
      default: return bwd_vec<IO, LN, kMaxVpl>(rows, c, dz, z, rstd, dx, s);
    }
  }
  if (rows > 0x7fffffff) return hipErrorInvalidValue;
  hipLaunchKernelGGL((norm_bwd_any<IO, LN>), dim3(unsigned(rows)), dim3(256), 0, s, dz, z, rstd, dx,
                     rows, cols);
  return hipGetLastError();
}
}  // namespace

hipError_t launch_norm_fwd(bool ln, bool bf16, int64_t rows, int64_t cols, float eps,
                           const void* x, void* z, float* rstd, bool vec_ok, hipStream_t s) {
  if (ln) return bf16 ? norm_fwd_t<BF16, true>(rows, cols, eps, x, z, rstd, vec_ok, s)
                      : norm_fwd_t<F32, true>(rows, cols, eps, x, z, rstd, vec_ok, s);
  return bf16 ? norm_fwd_t<BF16, false>(rows, cols, eps, x, z, rstd, vec_ok, s)
              : norm_fwd_t<F32, false>(rows, cols, eps, x, z, rstd, vec_ok, s);
}

hipError_t launch_norm_bwd(bool ln, bool bf16, int64_t rows, int64_t cols, const void* dz,
                           const void* z, const float* rstd, void* dx, bool vec_ok,
                           hipStream_t s) {
  if (ln) return bf16 ? norm_bwd_t<BF16, true>(rows, cols, dz, z, rstd, dx, vec_ok, s)
                      : norm_bwd_t<F32, true>(rows, cols, dz, z, rstd, dx, vec_ok, s);
  return bf16 ? norm_bwd_t<BF16, false>(rows, cols, dz, z, rstd, dx, vec_ok, s)
              : norm_bwd_t<F32, false>(rows, cols, dz, z, rstd, dx, vec_ok, s);
}

// ---------------------------------------------------------- measurement copy
__global__ __launch_bounds__(256) void copy16_kernel(const u32x4* __restrict__ src,
                                                     u32x4* __restrict__ dst, int64_t nvec,
                                                     const uint8_t* __restrict__ src_tail,
                                                     uint8_t* __restrict__ dst_tail, int tail) {
  constexpr int kU = 4;
  const int64_t base = int64_t(blockIdx.x) * (256 * kU) + threadIdx.x;
  u32x4 t[kU];
#pragma unroll
  for (int u = 0; u < kU; ++u) {
    const int64_t i = base + u * 256;
    if (i < nvec) t[u] = src[i];
  }
#pragma unroll
  for (int u = 0; u < kU; ++u) {
    const int64_t i = base + u * 256;
    if (i < nvec) dst[i] = t[u];
  }
  if (blockIdx.x == 0 && threadIdx.x < tail) dst_tail[threadIdx.x] = src_tail[threadIdx.x];
}

hipError_t launch_copy(const void* src, void* dst, int64_t bytes, hipStream_t s) {
  const int64_t nvec = bytes / 16;
  const int tail = int(bytes % 16);
  const int64_t blocks = (nvec + 1023) / 1024 > 0 ? (nvec + 1023) / 1024 : 1;
  if (blocks > 0x7fffffff) return hipErrorInvalidValue;
  hipLaunchKernelGGL(copy16_kernel, dim3(unsigned(blocks)), dim3(256), 0, s,
                     static_cast<const u32x4*>(src), static_cast<u32x4*>(dst), nvec,
                     static_cast<const uint8_t*>(src) + nvec * 16,
                     static_cast<uint8_t*>(dst) + nvec * 16, tail);
  return hipGetLastError();
}

}  // namespace lmbp
