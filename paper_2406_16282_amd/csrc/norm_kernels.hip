// MS-LN / MS-RMSNorm kernels for gfx950 (Sec. 5.2 Alg. 1; Appendix G Alg. 2, Alg. 3).
//
// Forward, per row x of width p: sigma = sqrt(p^-1 |H x|^2 + eps), z = H x / sigma,
// rstd = 1 / sigma, where H x = x - mean(x) (LN) or x (RMS). Backward from the saved
// output alone: dx = rstd * (H dz - z * p^-1 z^T dz).
//
// Fast path: 1, 2 or 4 waves per row (chosen from the row width), the row held in
// registers (thread t of a row holding 16-byte vectors t, t + 64*WPR, ...), so each
// tensor is read from HBM once and every statistic is a register pass plus a wave
// reduction (and one LDS exchange when a row spans several waves). The forward
// for rows of one wave runs persistent blocks that prefetch their next row. Rows that
// are not 16-byte aligned, or wider than 4 waves x 16 vectors, use a block-per-row
// path that re-reads the row for each pass.
//
// Numerics: LN accumulates x - x0 (x0 = the row's first element) so that rows
// with a large common offset do not lose the deviations to rounding; the centred
// values are (x - x0) - mean(x - x0), never x - mean(x) with mean(x) rounded.
// Variances are two-pass over the register-resident row.
#include "lmbp_device.hpp"
#include "lmbp_launch.hpp"

#include <atomic>

namespace lmbp {

#ifndef LMBP_NORM_NT
// Non-temporal loads (bit 0). Inputs are touched once per launch, so they stream past
// the caches (cold, default-policy loads were slower).
#define LMBP_NORM_NT 1
#endif
#ifndef LMBP_NORM_FWD_NT
#define LMBP_NORM_FWD_NT LMBP_NORM_NT  // the forward kernel's policy
#endif
#ifndef LMBP_NORM_BWD_NT
#define LMBP_NORM_BWD_NT LMBP_NORM_NT  // the backward kernel's policy
#endif
#ifndef LMBP_NORM_STORE_CPOL
// Cache policy of the 16-byte stores (buffer instructions): non-temporal (2). Stores at
// device scope (sc1), with or without nt, were slower here when the outputs are cold.
#define LMBP_NORM_STORE_CPOL 2
#endif
constexpr bool kFwdNtLoad = (LMBP_NORM_FWD_NT & 1) != 0;
constexpr bool kBwdNtLoad = (LMBP_NORM_BWD_NT & 1) != 0;

// Threads per block of the register-tile path: 256, or one row of WPR waves when
// that is wider (WPR = 8).
template <int WPR>
constexpr int norm_block() { return WPR * kWave > 256 ? WPR * kWave : 256; }

// Sum over the WPR waves that share a row (the row's waves consecutive in the
// block). Each LDS slot is written by one call per kernel, so one barrier
// suffices. Every thread of the block must call it.
template <int WPR, int NS>
__device__ inline void row_sums(float (&v)[NS], float (*red)[norm_block<WPR>() / kWave]) {
#pragma unroll
  for (int i = 0; i < NS; ++i) v[i] = wave_sum(v[i]);
  if constexpr (WPR > 1) {
    const int wave = threadIdx.x / kWave;
    if ((threadIdx.x & (kWave - 1)) == 0) {
#pragma unroll
      for (int i = 0; i < NS; ++i) red[i][wave] = v[i];
    }
    __syncthreads();
    const int first = (wave / WPR) * WPR;
#pragma unroll
    for (int i = 0; i < NS; ++i) {
      float t = 0.0f;
#pragma unroll
      for (int k = 0; k < WPR; ++k) t += red[i][first + k];
      v[i] = t;
    }
  }
}

// Register-tile path: WPR waves per row, thread t of the row (0 <= t < 64*WPR)
// holding vectors t, t + 64*WPR, ... (VPL of them). Rows start on 16-byte
// boundaries (checked by the host).
template <class IO, bool LN, int VPL, int WPR>
__global__ __launch_bounds__(norm_block<WPR>()) void norm_fwd_vec(const void* x, void* z,
                                                                  float* __restrict__ rstd,
                                                                  int64_t rows, int cols, float eps) {
  constexpr int E = IO::kPerVec;
  constexpr int TPR = kWave * WPR;
  constexpr int RPB = norm_block<WPR>() / TPR;
  __shared__ float red[2][norm_block<WPR>() / kWave];
  const int t = threadIdx.x % TPR;
  const int64_t row = int64_t(blockIdx.x) * RPB + wave_in_block() / WPR;
  const bool active = row < rows;
  if constexpr (WPR == 1) {
    if (!active) return;  // no barriers in the single-wave path
  }
  const int nv = cols / E;
  const int64_t vbase = row * nv;

  u32x4 v[VPL];
#pragma unroll
  for (int j = 0; j < VPL; ++j) {
    const int idx = j * TPR + t;
    v[j] = (active && idx < nv) ? ldg16<kFwdNtLoad>(x, vbase + idx) : u32x4{0u, 0u, 0u, 0u};
  }

  float pivot = 0.0f, mean_d = 0.0f;
  if constexpr (LN) {
    pivot = active ? IO::load1(x, row * int64_t(cols)) : 0.0f;
    float s[1] = {0.0f};
#pragma unroll
    for (int j = 0; j < VPL; ++j) {
      if (j * TPR + t < nv) {
        float f[E];
        IO::unpack(v[j], f);
#pragma unroll
        for (int e = 0; e < E; ++e) s[0] += f[e] - pivot;
      }
    }
    row_sums<WPR>(s, &red[0]);
    mean_d = s[0] / float(cols);
  }

  float q[1] = {0.0f};
#pragma unroll
  for (int j = 0; j < VPL; ++j) {
    if (j * TPR + t < nv) {
      float f[E];
      IO::unpack(v[j], f);
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const float c = LN ? (f[e] - pivot) - mean_d : f[e];
        q[0] = __builtin_fmaf(c, c, q[0]);
      }
    }
  }
  row_sums<WPR>(q, &red[1]);
  const float rs = rsqrtf(q[0] / float(cols) + eps);
  if (!active) return;

  if (z != nullptr) {   // null z: statistics only (the pre-pass of the fused norm-linear)
#pragma unroll
    for (int j = 0; j < VPL; ++j) {
      opaque(v[j]);
      const int idx = j * TPR + t;
      if (idx < nv) {
        float f[E];
        IO::unpack(v[j], f);
#pragma unroll
        for (int e = 0; e < E; ++e) f[e] = (LN ? (f[e] - pivot) - mean_d : f[e]) * rs;
        stb16<LMBP_NORM_STORE_CPOL>(vec_rsrc(z, vbase, nv), idx, IO::pack(f));
      }
    }
  }
  if (t == 0) rstd[row] = rs;
}

template <class IO, bool LN, int VPL, int WPR>
__global__ __launch_bounds__(norm_block<WPR>()) void norm_bwd_vec(const void* dz, const void* z,
                                                                  const float* __restrict__ rstd,
                                                                  void* dx, int64_t rows, int cols) {
  constexpr int E = IO::kPerVec;
  constexpr int TPR = kWave * WPR;
  constexpr int RPB = norm_block<WPR>() / TPR;
  __shared__ float red[2][norm_block<WPR>() / kWave];
  const int t = threadIdx.x % TPR;
  const int64_t row = int64_t(blockIdx.x) * RPB + wave_in_block() / WPR;
  const bool active = row < rows;
  if constexpr (WPR == 1) {
    if (!active) return;
  }
  const int nv = cols / E;
  const int64_t vbase = row * nv;

  u32x4 vg[VPL], vz[VPL];
#pragma unroll
  for (int j = 0; j < VPL; ++j) {
    const int idx = j * TPR + t;
    const bool ok = active && idx < nv;
    vg[j] = ok ? ldg16<kBwdNtLoad>(dz, vbase + idx) : u32x4{0u, 0u, 0u, 0u};
    vz[j] = ok ? ldg16<kBwdNtLoad>(z, vbase + idx) : u32x4{0u, 0u, 0u, 0u};
  }
  const float rs = active ? rstd[row] : 0.0f;

  // Zero padding contributes nothing to either sum.
  float s[2] = {0.0f, 0.0f};
#pragma unroll
  for (int j = 0; j < VPL; ++j) {
    float g[E], zz[E];
    IO::unpack(vg[j], g);
    IO::unpack(vz[j], zz);
#pragma unroll
    for (int e = 0; e < E; ++e) {
      if constexpr (LN) s[0] += g[e];
      s[1] = __builtin_fmaf(zz[e], g[e], s[1]);
    }
  }
  row_sums<WPR>(s, red);
  if (!active) return;
  const float a = LN ? s[0] / float(cols) : 0.0f;
  const float b = s[1] / float(cols);

#pragma unroll
  for (int j = 0; j < VPL; ++j) {
    opaque(vg[j]);
    opaque(vz[j]);
    const int idx = j * TPR + t;
    if (idx < nv) {
      float g[E], zz[E];
      IO::unpack(vg[j], g);
      IO::unpack(vz[j], zz);
#pragma unroll
      for (int e = 0; e < E; ++e) g[e] = rs * __builtin_fmaf(-zz[e], b, g[e] - a);
      stb16<LMBP_NORM_STORE_CPOL>(vec_rsrc(dx, vbase, nv), idx, IO::pack(g));
    }
  }
}

#ifndef LMBP_NORM_FWD_PIPE_WPR
// The forward takes the persistent form below for rows of at most this many waves (0:
// never). Measured: one wave per row (ViT-B, 768 wide) 11% faster; four waves per row
// (LLaMA, 4096 and 5120 wide) 6% slower, and the backward slower in both cases.
#define LMBP_NORM_FWD_PIPE_WPR 1
#endif

// Register-tile path, persistent form (forward): each block walks row groups
// g = blockIdx.x, blockIdx.x + gridDim.x, ... (a group = the block's RPB rows), with the
// next group's loads issued before the current group's reductions and stores, which
// hides the load latency of short rows. Every access is a buffer instruction over the
// row (an inactive row has an empty resource, padding lanes are out of range), so the
// loop has no memory branches and the compiler waits only for the loads it needs. The
// LDS slots alternate between consecutive groups: a wave can be at most one barrier
// ahead of another.
__device__ inline __amdgpu_buffer_rsrc_t row_rsrc(const void* base, int64_t first_byte, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(
      const_cast<char*>(static_cast<const char*>(base)) + first_byte, 0, bytes, 0x00020000);
}
constexpr uint32_t kNoLane = 0x80000000u;   // an offset beyond every resource

template <class IO, bool LN, int VPL, int WPR>
__global__ __launch_bounds__(norm_block<WPR>()) void norm_fwd_pipe(const void* x, void* z,
                                                                   float* __restrict__ rstd,
                                                                   int64_t rows, int cols, float eps) {
  constexpr int E = IO::kPerVec;
  constexpr int TPR = kWave * WPR;
  constexpr int RPB = norm_block<WPR>() / TPR;
  constexpr int kLoadPol = kFwdNtLoad ? 2 : 0;
  __shared__ float red[2][2][norm_block<WPR>() / kWave];
  const int t = threadIdx.x % TPR;
  const int sub = wave_in_block() / WPR;
  const int nv = cols / E;
  const int64_t groups = (rows + RPB - 1) / RPB;

  auto load = [&](int64_t g, u32x4 (&v)[VPL], float& pivot) {
    const int64_t row = g * RPB + sub;
    const bool active = g < groups && row < rows;
    const auto r = row_rsrc(x, active ? row * nv * 16 : 0, active ? nv * 16 : 0);
#pragma unroll
    for (int j = 0; j < VPL; ++j)
      v[j] = __builtin_amdgcn_raw_buffer_load_b128(r, uint32_t(j * TPR + t) * 16, 0, kLoadPol);
    if constexpr (LN) {
      float f[E];
      IO::unpack(__builtin_amdgcn_raw_buffer_load_b128(r, 0, 0, kLoadPol), f);
      pivot = f[0];
    }
  };

  u32x4 v[VPL], vn[VPL];
  float pivot = 0.0f, pivot_n = 0.0f;
  int par = 0;
  load(blockIdx.x, v, pivot);
  for (int64_t g = blockIdx.x; g < groups; g += gridDim.x, par ^= 1) {
    load(g + gridDim.x, vn, pivot_n);
    const int64_t row = g * RPB + sub;
    const bool active = row < rows;

    float mean_d = 0.0f;
    if constexpr (LN) {
      float s[1] = {0.0f};
#pragma unroll
      for (int j = 0; j < VPL; ++j) {
        float f[E];
        IO::unpack(v[j], f);
        const bool in = j * TPR + t < nv;
#pragma unroll
        for (int e = 0; e < E; ++e) s[0] += in ? f[e] - pivot : 0.0f;
      }
      row_sums<WPR>(s, &red[par][0]);
      mean_d = s[0] / float(cols);
    }
    float q[1] = {0.0f};
#pragma unroll
    for (int j = 0; j < VPL; ++j) {
      float f[E];
      IO::unpack(v[j], f);
      const bool in = j * TPR + t < nv;
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const float c = in ? (LN ? (f[e] - pivot) - mean_d : f[e]) : 0.0f;
        q[0] = __builtin_fmaf(c, c, q[0]);
      }
    }
    row_sums<WPR>(q, &red[par][1]);
    const float rs = rsqrtf(q[0] / float(cols) + eps);
    // a null z (statistics only) gets an empty resource: its stores are dropped
    const auto rz = row_rsrc(z, active ? row * nv * 16 : 0, (active && z != nullptr) ? nv * 16 : 0);
#pragma unroll
    for (int j = 0; j < VPL; ++j) {
      opaque(v[j]);
      float f[E];
      IO::unpack(v[j], f);
#pragma unroll
      for (int e = 0; e < E; ++e) f[e] = (LN ? (f[e] - pivot) - mean_d : f[e]) * rs;
      __builtin_amdgcn_raw_buffer_store_b128(IO::pack(f), rz, uint32_t(j * TPR + t) * 16, 0,
                                             LMBP_NORM_STORE_CPOL);
    }
    const auto rr = row_rsrc(rstd, active ? row * 4 : 0, active ? 4 : 0);
    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(rs), rr, t == 0 ? 0u : kNoLane, 0, 0);
#pragma unroll
    for (int j = 0; j < VPL; ++j) v[j] = vn[j];
    pivot = pivot_n;
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
  if (z != nullptr) {
    for (int64_t k = tid; k < cols; k += blockDim.x) {
      const float f = IO::load1(x, base + k);
      IO::store1(z, base + k, (LN ? (f - pivot) - mean_d : f) * rs);
    }
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
#ifndef LMBP_NORM_TARGET_VPL
#define LMBP_NORM_TARGET_VPL 2  // preferred upper bound on vectors per thread
#endif
#ifndef LMBP_NORM_FWD_VPL
// The forward's target: 3 lets a 768-wide fp32 row (192 vectors) run on one wave with
// three vectors per thread, and with it the persistent form (9% faster than two waves of
// two vectors, a quarter of them idle); the backward was 3% slower that way.
#define LMBP_NORM_FWD_VPL 3
#endif
#ifndef LMBP_NORM_BWD_VPL
#define LMBP_NORM_BWD_VPL LMBP_NORM_TARGET_VPL  // the backward kernel's target
#endif
#ifndef LMBP_NORM_MAX_WPR
#define LMBP_NORM_MAX_WPR 4  // widest row group (waves per row)
#endif
static_assert(LMBP_NORM_MAX_WPR == 1 || LMBP_NORM_MAX_WPR == 2 || LMBP_NORM_MAX_WPR == 4 ||
                  LMBP_NORM_MAX_WPR == 8,
              "waves per row must be 1, 2, 4 or 8");

namespace {
// Launch shape of the register-tile path: WPR waves per row and VPL 16-byte
// vectors per thread, chosen from the row width in vectors (nv): the fewest waves
// per row that keep VPL within the direction's target (so registers stay low,
// occupancy high and many rows are in flight per CU); rows wider than that use
// the widest group with more vectors per thread, up to its capacity. Wider rows
// take the block-per-row path. {0, 0} stands for that path.
struct NormShape {
  int wpr, vpl;
};
constexpr int kVplSmall[] = {1, 2, 3, 4, 6, 8};
constexpr int kVplWide[] = {1, 2, 3, 4, 6, 8, 12, 16};

constexpr bool in_list(int v, const int* list, int n) {
  for (int i = 0; i < n; ++i)
    if (list[i] == v) return true;
  return false;
}

// Whether pick_shape can return (wpr, vpl) for the given target; only those
// shapes are instantiated.
constexpr bool reachable(int wpr, int vpl, int target) {
  if (wpr > LMBP_NORM_MAX_WPR) return false;
  if (in_list(vpl, kVplSmall, 6) && vpl <= target) return true;
  return wpr == LMBP_NORM_MAX_WPR && in_list(vpl, kVplWide, 8) && (wpr < 8 || vpl <= 8);
}

NormShape pick_shape(int64_t nv, int target) {
  for (int wpr = 1; wpr <= LMBP_NORM_MAX_WPR; wpr *= 2) {
    if (int64_t(kWave) * wpr * target < nv) continue;
    for (int v : kVplSmall)
      if (v <= target && int64_t(kWave) * wpr * v >= nv) return {wpr, v};
  }
  const int wpr = LMBP_NORM_MAX_WPR;
  for (int v : kVplWide) {
    if (wpr == 8 && v > 8) break;
    if (int64_t(kWave) * wpr * v >= nv) return {wpr, v};
  }
  return {0, 0};
}

// Every shape the selection could produce for some knob setting, in one list; the
// dispatchers below walk it at compile time and instantiate the reachable ones.
constexpr NormShape kShapes[] = {
    {1, 1}, {1, 2}, {1, 3}, {1, 4}, {1, 6}, {1, 8},
    {2, 1}, {2, 2}, {2, 3}, {2, 4}, {2, 6}, {2, 8}, {2, 12}, {2, 16},
    {4, 1}, {4, 2}, {4, 3}, {4, 4}, {4, 6}, {4, 8}, {4, 12}, {4, 16},
    {8, 1}, {8, 2}, {8, 3}, {8, 4}, {8, 6}, {8, 8}};
constexpr int kNumShapes = sizeof(kShapes) / sizeof(kShapes[0]);

// Blocks of the persistent form: those resident at once on the device (from the
// kernel's occupancy, queried once per kernel and device), at most one per row group.
// Any grid is correct; if the queries fail, one block per group.
template <auto Kernel>
int64_t persistent_grid(int block, int64_t groups) {
  constexpr int kMaxDevices = 64;
  static std::atomic<int64_t> resident[kMaxDevices];
  int device = 0;
  if (hipGetDevice(&device) != hipSuccess || device < 0 || device >= kMaxDevices) return groups;
  int64_t r = resident[device].load(std::memory_order_relaxed);
  if (r == 0) {
    int cus = 0, per_cu = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device) != hipSuccess ||
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, Kernel, block, 0) != hipSuccess ||
        cus <= 0 || per_cu <= 0)
      return groups;
    r = int64_t(cus) * per_cu;
    resident[device].store(r, std::memory_order_relaxed);
  }
  return groups < r ? groups : r;
}

template <class IO, bool LN, int I>
hipError_t fwd_dispatch(NormShape sh, int64_t rows, int cols, float eps, const void* x, void* z,
                        float* rstd, hipStream_t s) {
  if constexpr (I == kNumShapes) {
    return hipErrorNotSupported;
  } else {
    constexpr int W = kShapes[I].wpr, V = kShapes[I].vpl;
    if constexpr (reachable(W, V, LMBP_NORM_FWD_VPL)) {
      if (sh.wpr == W && sh.vpl == V) {
        constexpr int rpb = norm_block<W>() / (kWave * W);
        const int64_t blocks = (rows + rpb - 1) / rpb;
        if (blocks > 0x7fffffff) return hipErrorInvalidValue;
        if constexpr (W <= LMBP_NORM_FWD_PIPE_WPR) {
          const int64_t grid = persistent_grid<norm_fwd_pipe<IO, LN, V, W>>(norm_block<W>(), blocks);
          hipLaunchKernelGGL((norm_fwd_pipe<IO, LN, V, W>), dim3(unsigned(grid)), dim3(norm_block<W>()),
                             0, s, x, z, rstd, rows, cols, eps);
          return hipGetLastError();
        }
        hipLaunchKernelGGL((norm_fwd_vec<IO, LN, V, W>), dim3(unsigned(blocks)), dim3(norm_block<W>()),
                           0, s, x, z, rstd, rows, cols, eps);
        return hipGetLastError();
      }
    }
    return fwd_dispatch<IO, LN, I + 1>(sh, rows, cols, eps, x, z, rstd, s);
  }
}

template <class IO, bool LN, int I>
hipError_t bwd_dispatch(NormShape sh, int64_t rows, int cols, const void* dz, const void* z,
                        const float* rstd, void* dx, hipStream_t s) {
  if constexpr (I == kNumShapes) {
    return hipErrorNotSupported;
  } else {
    constexpr int W = kShapes[I].wpr, V = kShapes[I].vpl;
    if constexpr (reachable(W, V, LMBP_NORM_BWD_VPL)) {
      if (sh.wpr == W && sh.vpl == V) {
        constexpr int rpb = norm_block<W>() / (kWave * W);
        const int64_t blocks = (rows + rpb - 1) / rpb;
        if (blocks > 0x7fffffff) return hipErrorInvalidValue;
        hipLaunchKernelGGL((norm_bwd_vec<IO, LN, V, W>), dim3(unsigned(blocks)), dim3(norm_block<W>()),
                           0, s, dz, z, rstd, dx, rows, cols);
        return hipGetLastError();
      }
    }
    return bwd_dispatch<IO, LN, I + 1>(sh, rows, cols, dz, z, rstd, dx, s);
  }
}

template <class IO, bool LN>
hipError_t norm_fwd_t(int64_t rows, int64_t cols, float eps, const void* x, void* z, float* rstd,
                      bool vec_ok, hipStream_t s) {
  const NormShape sh = vec_ok ? pick_shape(cols / IO::kPerVec, LMBP_NORM_FWD_VPL) : NormShape{0, 0};
  if (sh.wpr != 0) return fwd_dispatch<IO, LN, 0>(sh, rows, int(cols), eps, x, z, rstd, s);
  if (rows > 0x7fffffff) return hipErrorInvalidValue;
  hipLaunchKernelGGL((norm_fwd_any<IO, LN>), dim3(unsigned(rows)), dim3(256), 0, s, x, z, rstd, rows,
                     cols, eps);
  return hipGetLastError();
}

template <class IO, bool LN>
hipError_t norm_bwd_t(int64_t rows, int64_t cols, const void* dz, const void* z, const float* rstd,
                      void* dx, bool vec_ok, hipStream_t s) {
  const NormShape sh = vec_ok ? pick_shape(cols / IO::kPerVec, LMBP_NORM_BWD_VPL) : NormShape{0, 0};
  if (sh.wpr != 0) return bwd_dispatch<IO, LN, 0>(sh, rows, int(cols), dz, z, rstd, dx, s);
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
// Plain streaming copy: one 16-byte vector per thread, non-temporal loads, and
// non-temporal stores at device scope (written through the XCD's L2 instead of left
// dirty there): the fastest plain copy measured on this GPU from 32 MiB up (at the
// hot-path kernels' sizes 1-3% faster than non-temporal stores alone).
__global__ __launch_bounds__(256) void copy16_kernel(const u32x4* __restrict__ src,
                                                     u32x4* __restrict__ dst, int64_t nvec,
                                                     const uint8_t* __restrict__ src_tail,
                                                     uint8_t* __restrict__ dst_tail, int tail) {
  const int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (i < nvec)   // the block's 256 vectors as the resource; only lanes inside the tensor store
    stb16<2 | 16>(vec_rsrc(dst, int64_t(blockIdx.x) * 256, 256), int(threadIdx.x), ldg16<true>(src, i));
  if (blockIdx.x == 0 && threadIdx.x < tail) dst_tail[threadIdx.x] = src_tail[threadIdx.x];
}

hipError_t launch_copy(const void* src, void* dst, int64_t bytes, hipStream_t s) {
  const int64_t nvec = bytes / 16;
  const int tail = int(bytes % 16);
  const int64_t blocks = nvec > 0 ? (nvec + 255) / 256 : 1;
  if (blocks > 0x7fffffff) return hipErrorInvalidValue;
  hipLaunchKernelGGL(copy16_kernel, dim3(unsigned(blocks)), dim3(256), 0, s,
                     static_cast<const u32x4*>(src), static_cast<u32x4*>(dst), nvec,
                     static_cast<const uint8_t*>(src) + nvec * 16,
                     static_cast<uint8_t*>(dst) + nvec * 16, tail);
  return hipGetLastError();
}

}  // namespace lmbp
