// Table-driven members of the ReLU-combination family (eq. relus_family for general
// k; Appendix I's ReGELU2-d is k = 2 with other constants), for gfx950.
//
// Forward: exact GELU or SiLU (fp32 arithmetic) and a k-bit code per element: the
// number of the 2^k - 1 thresholds strictly below x (each compared exactly, against
// the largest fp32 value not above it, rounded on the host). Codes are packed floor(32/k)
// per 32-bit word, least significant first (k = 1, 2, 3, 4). Backward: dx = dy *
// levels[code], the 2^k levels read from an LDS table.
//
// Tiling (k = 1, 2, 4): one 16-byte vector per lane (E = 4 or 8 elements, E*k code
// bits); the G = 32 / (E*k) lanes that share a code word shift their parts into place
// and OR them together with cross-lane shuffles, and the group's first lane stores the
// word.
//
// k = 3: ten codes per word (bits 3j .. 3j + 2, top two bits zero), so a word's codes
// do not fall on vector boundaries. A wave handles 640 elements (64 words): each lane
// converts whole vectors and writes their codes as bytes to the wave's LDS area, then
// lane l packs bytes 10 l .. 10 l + 9 into word l (coalesced stores). The backward
// stages the 64 words in LDS the same way and each element reads its 3 bits there.
#include "lmbp_device.hpp"
#include "act_math.hpp"
#include "lmbp_launch.hpp"

#include <type_traits>

namespace lmbp {

template <class IO, int BITS>
struct StepShape {
  static constexpr int E = IO::kPerVec;
  static constexpr int PART = E * BITS;          // code bits per vector
  static constexpr int G = 32 / PART;            // lanes per code word (1, 2, 4 or 8)
  static constexpr int TILE = kWave * E;         // elements per wave tile
  static constexpr int NT = (1 << BITS) - 1;     // thresholds
  static_assert(G >= 1 && G <= 8 && 32 % PART == 0, "unsupported code width");
};

template <int NT>
__device__ inline uint32_t count_below(float x, const StepTable& tab) {
  uint32_t c = 0;
#pragma unroll
  for (int i = 0; i < NT; ++i) c += uint32_t(x > tab.t[i]);
  return c;
}

template <int G>
__device__ inline uint32_t group_or(uint32_t v) {
#pragma unroll
  for (int off = 1; off < G; off <<= 1) v |= uint32_t(__shfl_xor(int(v), off, kWave));
  return v;
}

template <class IO, int ACT, int BITS>
__global__ __launch_bounds__(128) void stepact_fwd_kernel(const void* x, void* y,
                                                          uint32_t* __restrict__ codes, int64_t n,
                                                          int vec_ok, StepTable tab) {
  using S = StepShape<IO, BITS>;
  constexpr bool kPrecise = std::is_same<IO, F32>::value;
  constexpr int E = S::E;
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t wave = int64_t(blockIdx.x) * (blockDim.x / kWave) + (threadIdx.x / kWave);
  const int64_t base = wave * S::TILE;
  if (base >= n) return;

  if (vec_ok && base + S::TILE <= n) {
    const u32x4 v = ldg16<true>(x, base / E + lane);
    float f[E], o[E];
    IO::unpack(v, f);
    uint32_t part = 0;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      o[e] = act_value<ACT, kPrecise>(f[e]);
      part |= count_below<S::NT>(f[e], tab) << (BITS * e);
    }
    stg16<true>(y, base / E + lane, IO::pack(o));
    const uint32_t word = group_or<S::G>(S::G == 1 ? part : part << ((lane % S::G) * S::PART));
    if (lane % S::G == 0) codes[base * BITS / 32 + lane / S::G] = word;
    return;
  }

  // General path: partial last tile or unaligned pointers; one code word per lane.
  constexpr int PER = 32 / BITS;
  const int64_t end = (base + S::TILE < n) ? base + S::TILE : n;
  const int64_t w_end = (end + PER - 1) / PER;
  for (int64_t w = base / PER + lane; w < w_end; w += kWave) {
    uint32_t word = 0;
    for (int e = 0; e < PER; ++e) {
      const int64_t i = w * PER + e;
      if (i < n) {
        const float xv = IO::load1(x, i);
        IO::store1(y, i, act_value<ACT, kPrecise>(xv));
        word |= count_below<S::NT>(xv, tab) << (BITS * e);
      }
    }
    codes[w] = word;
  }
}

template <class IO, int BITS>
__global__ __launch_bounds__(128) void stepact_bwd_kernel(const void* dy,
                                                          const uint32_t* __restrict__ codes,
                                                          void* dx, int64_t n, int vec_ok,
                                                          StepTable tab) {
  using S = StepShape<IO, BITS>;
  constexpr int E = S::E;
  constexpr uint32_t kMask = (1u << BITS) - 1u;
  __shared__ float lv[1 << BITS];
  if (threadIdx.x < (1 << BITS)) lv[threadIdx.x] = tab.lv[threadIdx.x];
  __syncthreads();
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t wave = int64_t(blockIdx.x) * (blockDim.x / kWave) + (threadIdx.x / kWave);
  const int64_t base = wave * S::TILE;
  if (base >= n) return;

  if (vec_ok && base + S::TILE <= n) {
    const u32x4 v = ldg16<true>(dy, base / E + lane);
    const uint32_t part = codes[base * BITS / 32 + lane / S::G] >> ((lane % S::G) * S::PART);
    float f[E];
    IO::unpack(v, f);
#pragma unroll
    for (int e = 0; e < E; ++e) f[e] *= lv[(part >> (BITS * e)) & kMask];
    stg16<true>(dx, base / E + lane, IO::pack(f));
    return;
  }

  constexpr int PER = 32 / BITS;
  const int64_t end = (base + S::TILE < n) ? base + S::TILE : n;
  for (int64_t i = base + lane; i < end; i += kWave) {
    const uint32_t c = (codes[i / PER] >> (BITS * (i % PER))) & kMask;
    IO::store1(dx, i, IO::load1(dy, i) * lv[c]);
  }
}

// ------------------------------------------------------------------ k = 3
constexpr int kTile3 = 640;     // elements per wave: 64 words of 10 codes
constexpr int kWords3 = kTile3 / 10;

template <class IO, int ACT>
__global__ __launch_bounds__(128) void stepact3_fwd_kernel(const void* x, void* y,
                                                           uint32_t* __restrict__ codes, int64_t n,
                                                           int vec_ok, StepTable tab) {
  constexpr bool kPrecise = std::is_same<IO, F32>::value;
  constexpr int E = IO::kPerVec;
  constexpr int NV = kTile3 / E;   // vectors per wave tile
  __shared__ uint8_t lcodes[2][kTile3];
  const int lane = threadIdx.x & (kWave - 1);
  const int wv = threadIdx.x / kWave;
  const int64_t base = (int64_t(blockIdx.x) * 2 + wv) * kTile3;
  if (base >= n) return;

  if (vec_ok && base + kTile3 <= n) {
    uint8_t* lc = lcodes[wv];
    for (int v = lane; v < NV; v += kWave) {
      const u32x4 in = ldg16<true>(x, base / E + v);
      float f[E], o[E];
      IO::unpack(in, f);
#pragma unroll
      for (int e = 0; e < E; ++e) {
        o[e] = act_value<ACT, kPrecise>(f[e]);
        lc[v * E + e] = uint8_t(count_below<7>(f[e], tab));
      }
      stg16<true>(y, base / E + v, IO::pack(o));
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");   // every lane's bytes are in LDS
    uint32_t word = 0;
#pragma unroll
    for (int j = 0; j < 10; ++j) word |= uint32_t(lc[lane * 10 + j]) << (3 * j);
    codes[base / 10 + lane] = word;
    return;
  }

  // General path: partial last tile or unaligned pointers; one code word per lane.
  const int64_t end = (base + kTile3 < n) ? base + kTile3 : n;
  const int64_t w_end = (end + 9) / 10;
  for (int64_t w = base / 10 + lane; w < w_end; w += kWave) {
    uint32_t word = 0;
    for (int j = 0; j < 10; ++j) {
      const int64_t i = w * 10 + j;
      if (i < n) {
        const float xv = IO::load1(x, i);
        IO::store1(y, i, act_value<ACT, kPrecise>(xv));
        word |= count_below<7>(xv, tab) << (3 * j);
      }
    }
    codes[w] = word;
  }
}

template <class IO>
__global__ __launch_bounds__(128) void stepact3_bwd_kernel(const void* dy,
                                                           const uint32_t* __restrict__ codes,
                                                           void* dx, int64_t n, int vec_ok,
                                                           StepTable tab) {
  constexpr int E = IO::kPerVec;
  constexpr int NV = kTile3 / E;
  __shared__ float lv[8];
  __shared__ uint32_t lwords[2][kWords3];
  if (threadIdx.x < 8) lv[threadIdx.x] = tab.lv[threadIdx.x];
  __syncthreads();
  const int lane = threadIdx.x & (kWave - 1);
  const int wv = threadIdx.x / kWave;
  const int64_t base = (int64_t(blockIdx.x) * 2 + wv) * kTile3;
  if (base >= n) return;

  if (vec_ok && base + kTile3 <= n) {
    uint32_t* lw = lwords[wv];
    lw[lane] = codes[base / 10 + lane];
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");   // every lane's word is in LDS
    for (int v = lane; v < NV; v += kWave) {
      float f[E];
      IO::unpack(ldg16<true>(dy, base / E + v), f);
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const int i = v * E + e;
        f[e] *= lv[(lw[i / 10] >> (3 * (i % 10))) & 7u];
      }
      stg16<true>(dx, base / E + v, IO::pack(f));
    }
    return;
  }

  const int64_t end = (base + kTile3 < n) ? base + kTile3 : n;
  for (int64_t i = base + lane; i < end; i += kWave) {
    const uint32_t c = (codes[i / 10] >> (3 * (i % 10))) & 7u;
    IO::store1(dx, i, IO::load1(dy, i) * lv[c]);
  }
}

namespace {
int64_t step3_blocks(int64_t n) {
  const int64_t waves = (n + kTile3 - 1) / kTile3;
  return (waves + 1) / 2;  // 2 waves per 128-thread block
}

template <class IO, int ACT>
hipError_t fwd3(int64_t n, const void* x, void* y, uint32_t* codes, bool vec_ok,
                const StepTable& tab, hipStream_t s) {
  const int64_t blocks = step3_blocks(n);
  if (blocks > 0x7fffffff) return hipErrorInvalidValue;
  hipLaunchKernelGGL((stepact3_fwd_kernel<IO, ACT>), dim3(unsigned(blocks)), dim3(128), 0, s, x, y,
                     codes, n, int(vec_ok), tab);
  return hipGetLastError();
}

template <class IO>
hipError_t bwd3(int64_t n, const void* dy, const uint32_t* codes, void* dx, bool vec_ok,
                const StepTable& tab, hipStream_t s) {
  const int64_t blocks = step3_blocks(n);
  if (blocks > 0x7fffffff) return hipErrorInvalidValue;
  hipLaunchKernelGGL((stepact3_bwd_kernel<IO>), dim3(unsigned(blocks)), dim3(128), 0, s, dy, codes,
                     dx, n, int(vec_ok), tab);
  return hipGetLastError();
}

template <class IO>
int64_t step_blocks(int64_t n) {
  const int64_t waves = (n + int64_t(kWave) * IO::kPerVec - 1) / (int64_t(kWave) * IO::kPerVec);
  return (waves + 1) / 2;  // 2 waves per 128-thread block
}

template <class IO, int ACT, int BITS>
hipError_t fwd_t(int64_t n, const void* x, void* y, uint32_t* codes, bool vec_ok,
                 const StepTable& tab, hipStream_t s) {
  const int64_t blocks = step_blocks<IO>(n);
  if (blocks > 0x7fffffff) return hipErrorInvalidValue;
  hipLaunchKernelGGL((stepact_fwd_kernel<IO, ACT, BITS>), dim3(unsigned(blocks)), dim3(128), 0, s, x, y,
                     codes, n, int(vec_ok), tab);
  return hipGetLastError();
}

template <class IO, int BITS>
hipError_t bwd_t(int64_t n, const void* dy, const uint32_t* codes, void* dx, bool vec_ok,
                 const StepTable& tab, hipStream_t s) {
  const int64_t blocks = step_blocks<IO>(n);
  if (blocks > 0x7fffffff) return hipErrorInvalidValue;
  hipLaunchKernelGGL((stepact_bwd_kernel<IO, BITS>), dim3(unsigned(blocks)), dim3(128), 0, s, dy, codes,
                     dx, n, int(vec_ok), tab);
  return hipGetLastError();
}

template <class IO, int ACT>
hipError_t fwd_bits(int bits, int64_t n, const void* x, void* y, uint32_t* codes, bool vec_ok,
                    const StepTable& tab, hipStream_t s) {
  switch (bits) {
    case 1: return fwd_t<IO, ACT, 1>(n, x, y, codes, vec_ok, tab, s);
    case 2: return fwd_t<IO, ACT, 2>(n, x, y, codes, vec_ok, tab, s);
    case 3: return fwd3<IO, ACT>(n, x, y, codes, vec_ok, tab, s);
    case 4: return fwd_t<IO, ACT, 4>(n, x, y, codes, vec_ok, tab, s);
    default: return hipErrorInvalidValue;
  }
}

template <class IO>
hipError_t bwd_bits(int bits, int64_t n, const void* dy, const uint32_t* codes, void* dx,
                    bool vec_ok, const StepTable& tab, hipStream_t s) {
  switch (bits) {
    case 1: return bwd_t<IO, 1>(n, dy, codes, dx, vec_ok, tab, s);
    case 2: return bwd_t<IO, 2>(n, dy, codes, dx, vec_ok, tab, s);
    case 3: return bwd3<IO>(n, dy, codes, dx, vec_ok, tab, s);
    case 4: return bwd_t<IO, 4>(n, dy, codes, dx, vec_ok, tab, s);
    default: return hipErrorInvalidValue;
  }
}
}  // namespace

hipError_t launch_stepact_fwd(int act, int bits, bool bf16, int64_t n, const void* x, void* y,
                              uint32_t* codes, bool vec_ok, const StepTable& tab, hipStream_t s) {
  if (act == kGelu)
    return bf16 ? fwd_bits<BF16, kGelu>(bits, n, x, y, codes, vec_ok, tab, s)
                : fwd_bits<F32, kGelu>(bits, n, x, y, codes, vec_ok, tab, s);
  return bf16 ? fwd_bits<BF16, kSilu>(bits, n, x, y, codes, vec_ok, tab, s)
              : fwd_bits<F32, kSilu>(bits, n, x, y, codes, vec_ok, tab, s);
}

hipError_t launch_stepact_bwd(int bits, bool bf16, int64_t n, const void* dy, const uint32_t* codes,
                              void* dx, bool vec_ok, const StepTable& tab, hipStream_t s) {
  return bf16 ? bwd_bits<BF16>(bits, n, dy, codes, dx, vec_ok, tab, s)
              : bwd_bits<F32>(bits, n, dy, codes, dx, vec_ok, tab, s);
}

}  // namespace lmbp
