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
// Codes are counted by a linear pass over the thresholds for k <= 2 and by binary search
// over an LDS copy of the table for k = 3, 4.
//
// k = 3: ten codes per word (bits 3j .. 3j + 2, top two bits zero), so a word's codes
// do not fall on vector boundaries; five vectors are whole words, and the k = 3 kernels
// below tile by them.
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

// The same count by binary search over the increasing thresholds (duplicates, which
// the round-down can produce, are counted alike): the first probe is the middle
// threshold, a kernel argument; the others read the lane's own entry of an LDS copy of
// the table. k - 1 LDS reads per element instead of 2^k - 1 compares.
template <int BITS>
__device__ inline uint32_t search_below(float x, const StepTable& tab, const float* lt) {
  constexpr uint32_t H = 1u << (BITS - 1);
  uint32_t c = (x > tab.t[H - 1]) ? H : 0u;
#pragma unroll
  for (uint32_t step = H / 2; step >= 1; step /= 2) c += (x > lt[c + step - 1]) ? step : 0u;
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
  constexpr bool kSearch = BITS >= 3;
  __shared__ float lt[16];
  if constexpr (kSearch) {
    if (threadIdx.x < S::NT) lt[threadIdx.x] = tab.t[threadIdx.x];
    __syncthreads();
  }
  auto code = [&](float v) {
    if constexpr (kSearch) return search_below<BITS>(v, tab, lt);
    else return count_below<S::NT>(v, tab);
  };
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
      part |= code(f[e]) << (BITS * e);
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
        word |= code(xv) << (BITS * e);
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
// Ten codes per word: 5 vectors (5 E elements) are E / 2 whole words. A wave tile is 64 x 5
// vectors. Forward, phase 1 (coalesced, vector j * 64 + lane): activation, y stored, and
// the vector's E codes as one 3E-bit part written to the wave's LDS area; phase 2: lane l
// reads the parts of vectors 5 l .. 5 l + 4 (odd stride: no bank conflicts), which are
// exactly words (E / 2) l .. (E / 2) l + E / 2 - 1, and stores them with one vector store.
// Backward: the tile's words are staged in LDS, and a vector's 3E code bits, which start
// at bit 3 (vE mod 10) of word vE / 10 and may run into the next word, come from two reads.
constexpr int kVec3 = 5;

template <class IO>
struct Tile3 {
  static constexpr int E = IO::kPerVec;
  static constexpr int TILE = kWave * kVec3 * E;   // elements per wave tile
  static constexpr int WPL = kVec3 * E / 10;       // code words per lane
  static constexpr int WORDS = kWave * WPL;        // code words per wave tile
  static constexpr int PART = 3 * E;               // code bits per vector
};

// Word i (30 bits) of the concatenation of the 5 parts (part j at bit PART j).
template <int PART, int I>
__device__ inline uint32_t word_of_parts(const uint32_t (&p)[kVec3]) {
  uint32_t w = 0;
#pragma unroll
  for (int j = 0; j < kVec3; ++j) {
    const int sh = PART * j - 30 * I;   // position of part j relative to the word's bit 0
    if (sh > -PART && sh < 30) w |= sh >= 0 ? p[j] << sh : p[j] >> -sh;
  }
  return w & 0x3FFFFFFFu;
}

template <class IO, int ACT>
__global__ __launch_bounds__(128) void stepact3_fwd_kernel(const void* x, void* y,
                                                           uint32_t* __restrict__ codes, int64_t n,
                                                           int vec_ok, StepTable tab) {
  using T3 = Tile3<IO>;
  constexpr bool kPrecise = std::is_same<IO, F32>::value;
  constexpr int E = T3::E;
  __shared__ float lt[8];
  __shared__ uint32_t lparts[2][kWave * kVec3];
  if (threadIdx.x < 7) lt[threadIdx.x] = tab.t[threadIdx.x];
  __syncthreads();
  const int lane = threadIdx.x & (kWave - 1);
  const int wv = threadIdx.x / kWave;
  const int64_t base = (int64_t(blockIdx.x) * 2 + wv) * T3::TILE;
  if (base >= n) return;

  if (vec_ok && base + T3::TILE <= n) {
    uint32_t* lp = lparts[wv];
#pragma unroll
    for (int j = 0; j < kVec3; ++j) {
      const int v = j * kWave + lane;
      const u32x4 in = ldg16<true>(x, base / E + v);
      float f[E], o[E];
      IO::unpack(in, f);
      uint32_t part = 0;
#pragma unroll
      for (int e = 0; e < E; ++e) {
        o[e] = act_value<ACT, kPrecise>(f[e]);
        part |= search_below<3>(f[e], tab, lt) << (3 * e);
      }
      stg16<true>(y, base / E + v, IO::pack(o));
      lp[v] = part;
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");   // the wave's parts are in LDS
    uint32_t p[kVec3];
#pragma unroll
    for (int j = 0; j < kVec3; ++j) p[j] = lp[kVec3 * lane + j];
    uint32_t* cw = codes + base / 10 + T3::WPL * lane;
    if constexpr (T3::WPL == 4) {
      u32x4 w;
      w[0] = word_of_parts<T3::PART, 0>(p);
      w[1] = word_of_parts<T3::PART, 1>(p);
      w[2] = word_of_parts<T3::PART, 2>(p);
      w[3] = word_of_parts<T3::PART, 3>(p);
      *reinterpret_cast<u32x4*>(cw) = w;
    } else {
      static_assert(T3::WPL == 2, "fp32: two words per lane");
      uint2 w;
      w.x = word_of_parts<T3::PART, 0>(p);
      w.y = word_of_parts<T3::PART, 1>(p);
      *reinterpret_cast<uint2*>(cw) = w;
    }
    return;
  }

  // General path: partial last tile or unaligned pointers; one code word per lane.
  const int64_t end = (base + T3::TILE < n) ? base + T3::TILE : n;
  const int64_t w_end = (end + 9) / 10;
  for (int64_t w = base / 10 + lane; w < w_end; w += kWave) {
    uint32_t word = 0;
    for (int j = 0; j < 10; ++j) {
      const int64_t i = w * 10 + j;
      if (i < n) {
        const float xv = IO::load1(x, i);
        IO::store1(y, i, act_value<ACT, kPrecise>(xv));
        word |= search_below<3>(xv, tab, lt) << (3 * j);
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
  using T3 = Tile3<IO>;
  constexpr int E = T3::E;
  __shared__ float lv[8];
  __shared__ uint32_t lwords[2][T3::WORDS + 1];
  if (threadIdx.x < 8) lv[threadIdx.x] = tab.lv[threadIdx.x];
  __syncthreads();
  const int lane = threadIdx.x & (kWave - 1);
  const int wv = threadIdx.x / kWave;
  const int64_t base = (int64_t(blockIdx.x) * 2 + wv) * T3::TILE;
  if (base >= n) return;

  if (vec_ok && base + T3::TILE <= n) {
    // The gradient vectors are requested first, so their latency overlaps the staging of
    // the code words.
    u32x4 g[kVec3];
#pragma unroll
    for (int j = 0; j < kVec3; ++j) g[j] = ldg16<true>(dy, base / E + j * kWave + lane);
    uint32_t* lw = lwords[wv];
#pragma unroll
    for (int i = 0; i < T3::WPL; ++i) lw[i * kWave + lane] = codes[base / 10 + i * kWave + lane];
    if (lane == 0) lw[T3::WORDS] = 0u;   // read (and discarded) by the last vector
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");   // the tile's words are in LDS
#pragma unroll
    for (int j = 0; j < kVec3; ++j) {
      const int v = j * kWave + lane;
      const int first = v * E;              // element offset in the tile
      const int w0 = first / 10, o = first % 10;
      const uint64_t pair = (uint64_t(lw[w0 + 1]) << 30) | (lw[w0] & 0x3FFFFFFFu);
      const uint32_t bits = uint32_t(pair >> (3 * o));
      float f[E];
      IO::unpack(g[j], f);
#pragma unroll
      for (int e = 0; e < E; ++e) f[e] *= lv[(bits >> (3 * e)) & 7u];
      stg16<true>(dx, base / E + v, IO::pack(f));
    }
    return;
  }

  const int64_t end = (base + T3::TILE < n) ? base + T3::TILE : n;
  for (int64_t i = base + lane; i < end; i += kWave) {
    const uint32_t c = (codes[i / 10] >> (3 * (i % 10))) & 7u;
    IO::store1(dx, i, IO::load1(dy, i) * lv[c]);
  }
}

namespace {
template <class IO>
int64_t step3_blocks(int64_t n) {
  const int64_t waves = (n + Tile3<IO>::TILE - 1) / Tile3<IO>::TILE;
  return (waves + 1) / 2;  // 2 waves per 128-thread block
}

template <class IO, int ACT>
hipError_t fwd3(int64_t n, const void* x, void* y, uint32_t* codes, bool vec_ok,
                const StepTable& tab, hipStream_t s) {
  const int64_t blocks = step3_blocks<IO>(n);
  if (blocks > 0x7fffffff) return hipErrorInvalidValue;
  hipLaunchKernelGGL((stepact3_fwd_kernel<IO, ACT>), dim3(unsigned(blocks)), dim3(128), 0, s, x, y,
                     codes, n, int(vec_ok), tab);
  return hipGetLastError();
}

template <class IO>
hipError_t bwd3(int64_t n, const void* dy, const uint32_t* codes, void* dx, bool vec_ok,
                const StepTable& tab, hipStream_t s) {
  const int64_t blocks = step3_blocks<IO>(n);
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
