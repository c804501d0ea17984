// ReGELU2 / ReSiLU2 kernels for gfx950 (Sec. 4.2, eq. relus_family with k = 2;
// constants from Appendix E).
//
// Forward: y = GELU(x) or SiLU(x) (exact function, fp32 arithmetic) and a 2-bit
// segment code per element, packed 16 codes per 32-bit word, least significant
// bits first. Backward: dx = dy * slope[code], slope = (0, a1, a1 + a2, 1).
//
// Layout of one wave's tile (fast path): lane l holds vectors j = 0..VPL-1 at
// vector index tile_vec + j*64 + l, so every load and store instruction of the
// wave covers 1 KiB of contiguous memory. A vector carries 4 (fp32) or 8 (bf16)
// elements, i.e. 8 or 16 code bits; G = 4 or 2 neighbouring lanes hold the parts
// of one code word. With one vector per lane (fp32, and the bf16 SwiGLU kernels) the
// G lanes of a group shift their parts into place and OR them; with VPL a multiple of
// G, each lane packs its G parts for G consecutive vectors into one
// 32-bit value and the group transposes them with DPP quad permutes, after which
// lane q of a group owns the complete word of vector (G*m + q): the word stores of
// a wave are then contiguous too.
#include "lmbp_device.hpp"
#include "act_codes.hpp"
#include "act_math.hpp"
#include "lmbp_launch.hpp"

#ifndef LMBP_ACT_VPL
// 16-byte vectors per lane in one wave tile, bf16 storage (1, or a multiple of the 2
// lanes that share a code word). Small tiles mean many short-lived waves, which
// measured best; one vector was 2-6% slower.
#define LMBP_ACT_VPL 2
#endif
#ifndef LMBP_ACT_VPL_F32
// fp32 storage: one vector per lane (four lanes share a code word). Measured against four
// (one code word per lane): ViT-B fp32 pair 4.48 vs 4.31 TB/s, an [8192 x 11008] fp32 pair
// 6.47 vs 6.32 TB/s (backward 8% faster, forward 3% slower).
#define LMBP_ACT_VPL_F32 1
#endif
#ifndef LMBP_GLU_VPL
// The same for the SwiGLU kernels with bf16 storage (fp32 keeps the activation
// kernels' tile). They move three (forward) or five (backward) tensors per element, so
// one vector per lane already keeps enough bytes in flight and the shorter waves pay:
// the LLaMA-7B pair streams 3-4% faster than with two.
#define LMBP_GLU_VPL 1
#endif
#ifndef LMBP_GLU_STORE_CPOL
#define LMBP_GLU_STORE_CPOL LMBP_ACT_STORE_CPOL
#endif
#ifndef LMBP_ACT_BLOCK
#define LMBP_ACT_BLOCK 128  // threads per block (a multiple of 64)
#endif
#ifndef LMBP_ACT_BLOCK_F32
// fp32 storage: one-wave blocks (one vector per lane, so a wave moves only 1 KiB per
// tensor). Measured against 128 threads, cold: ViT-B fp32 ReGELU2 pair 4.68 vs 4.45 TB/s,
// LLaMA-7B-gate-sized fp32 ReSiLU2 pair (2048 x 11008) 6.44 vs 6.19 TB/s.
#define LMBP_ACT_BLOCK_F32 64
#endif
static_assert(LMBP_ACT_BLOCK_F32 <= LMBP_ACT_BLOCK, "fp32 blocks within the launch bounds");
#ifndef LMBP_ACT_NT
// Non-temporal data loads (bit 0) / code-word stores (bit 2) / code-word loads (bit 3).
// Inputs are touched once, so they stream; the 4-byte code-word accesses are faster
// with the default policy.
#define LMBP_ACT_NT 1
#endif
#ifndef LMBP_ACT_STORE_CPOL
// Cache policy of the 16-byte data stores (buffer instructions): non-temporal at device
// scope (nt sc1 = 2 | 16), written through the XCD's L2 instead of left dirty for the
// end-of-kernel write-back; measured 1.5-3% faster than non-temporal alone, cold.
#define LMBP_ACT_STORE_CPOL (2 | 16)
#endif

namespace lmbp {

constexpr bool kActNtLoad = (LMBP_ACT_NT & 1) != 0;
constexpr bool kActNtCodeStore = (LMBP_ACT_NT & 4) != 0;
constexpr bool kActNtCodeLoad = (LMBP_ACT_NT & 8) != 0;

// Store the code words of one wave tile. part[j] holds the 2E code bits of this
// lane's vector j (vector index tile_vec + j*64 + lane), G lanes sharing a word.
//   VPL == 1: the G lanes of a group shift their parts into place and OR them
//   together with one or two DPP steps; the group's first lane stores the word.
//   VPL a multiple of G: each lane packs its parts of G consecutive vectors into one
//   32-bit value and the group transposes them with DPP quad permutes (step s: lane q
//   sends part (q - s) mod G and receives, from lane (q + s) mod G, that lane's part
//   for vector G*m + q), so every lane stores a whole word and the stores of a wave
//   are contiguous.
template <class IO, int VPL>
__device__ inline void store_tile_codes(uint32_t* __restrict__ codes, int64_t wbase,
                                        const uint32_t (&part)[VPL], int lane) {
  constexpr int E = IO::kPerVec;
  constexpr int G = 16 / E;
  constexpr int PART = 2 * E;
  static_assert(VPL == 1 || VPL % G == 0, "VPL must be 1 or a multiple of the lane group");
  const int q = lane % G;
  if constexpr (VPL == 1) {
    uint32_t word = part[0] << (q * PART);
    word |= group_rotate<G, 1>(word);
    if constexpr (G == 4) word |= group_rotate<4, 2>(word);
    if (q == 0) {
      if constexpr (kActNtCodeStore) __builtin_nontemporal_store(word, codes + wbase + lane / G);
      else codes[wbase + lane / G] = word;
    }
  } else {
#pragma unroll
    for (int m = 0; m < VPL / G; ++m) {
      uint32_t packed = 0;
#pragma unroll
      for (int t = 0; t < G; ++t) packed |= part[G * m + t] << (t * PART);
      uint32_t word = 0;
#pragma unroll
      for (int s = 0; s < G; ++s) {
        const uint32_t send = __builtin_amdgcn_alignbit(packed, packed, uint32_t(((q - s + G) % G) * PART));
        uint32_t recv;
        if constexpr (G == 2) {
          recv = (s == 0) ? send : group_rotate<2, 1>(send);
        } else {
          recv = (s == 0) ? send : (s == 1) ? group_rotate<4, 1>(send)
               : (s == 2) ? group_rotate<4, 2>(send) : group_rotate<4, 3>(send);
        }
        const uint32_t mask = (PART == 32) ? 0xffffffffu : ((1u << PART) - 1u);
        word |= (recv & mask) << (((q + s) % G) * PART);
      }
      uint32_t* cw = codes + wbase + int64_t(G * m + q) * (kWave / G) + lane / G;
      if constexpr (kActNtCodeStore) __builtin_nontemporal_store(word, cw);
      else *cw = word;
    }
  }
}

// Load, for each of this lane's VPL vectors, the code bits of that vector (the
// word shared by the lane group, shifted to this lane's part).
template <class IO, int VPL>
__device__ inline void load_tile_codes(const uint32_t* __restrict__ codes, int64_t wbase,
                                       uint32_t (&part)[VPL], int lane) {
  constexpr int G = 16 / IO::kPerVec;
  constexpr int PART = 2 * IO::kPerVec;
#pragma unroll
  for (int j = 0; j < VPL; ++j) {
    const uint32_t* cw = codes + wbase + j * (kWave / G) + lane / G;
    uint32_t w;
    if constexpr (kActNtCodeLoad) w = __builtin_nontemporal_load(cw);
    else w = *cw;
    part[j] = w >> ((lane % G) * PART);
  }
}

// -------------------------------------------------------------------- kernels
template <class IO, int ACT, int VPL>
__global__ __launch_bounds__(LMBP_ACT_BLOCK) void act_fwd_kernel(const void* x, void* y,
                                                      uint32_t* __restrict__ codes,
                                                      int64_t n, int vec_ok) {
  using A = ActOf<ACT>;
  constexpr bool kPrecise = std::is_same<IO, F32>::value;
  constexpr int E = IO::kPerVec;      // elements per 16-byte vector
  constexpr int TILE = kWave * VPL * E;

  const int lane = threadIdx.x & (kWave - 1);
  const int64_t wave = int64_t(blockIdx.x) * (blockDim.x / kWave) + wave_in_block();
  const int64_t base = wave * TILE;
  if (base >= n) return;

  if (vec_ok && base + TILE <= n) {
    const int64_t vbase = base / E;
    u32x4 in[VPL];
#pragma unroll
    for (int j = 0; j < VPL; ++j) in[j] = ldg16<kActNtLoad>(x, vbase + j * kWave + lane);

    uint32_t part[VPL];
#pragma unroll
    for (int j = 0; j < VPL; ++j) {
      float f[E], o[E];
      IO::unpack(in[j], f);
#pragma unroll
      for (int e = 0; e < E; ++e) o[e] = act_value<ACT, kPrecise>(f[e]);
      part[j] = codes_of<A>(f);
      stb16<LMBP_ACT_STORE_CPOL>(vec_rsrc(y, vbase, VPL * kWave), j * kWave + lane, IO::pack(o));
    }

    store_tile_codes<IO, VPL>(codes, base / 16, part, lane);
    return;
  }

  // General path: the partial last tile, or pointers that are not 16-byte aligned.
  const int64_t end = (base + TILE < n) ? base + TILE : n;
  const int64_t w_end = (end + 15) / 16;
  for (int64_t w = base / 16 + lane; w < w_end; w += kWave) {
    uint32_t word = 0;
    for (int e = 0; e < 16; ++e) {
      const int64_t i = w * 16 + e;
      if (i < n) {
        const float xv = IO::load1(x, i);
        IO::store1(y, i, act_value<ACT, kPrecise>(xv));
        word |= seg_code<A>(xv) << (2 * e);
      }
    }
    codes[w] = word;
  }
}

template <class IO, int ACT, int VPL>
__global__ __launch_bounds__(LMBP_ACT_BLOCK) void act_bwd_kernel(const void* dy,
                                                      const uint32_t* __restrict__ codes,
                                                      void* dx, int64_t n, int vec_ok) {
  using A = ActOf<ACT>;
  constexpr int E = IO::kPerVec;
  constexpr int TILE = kWave * VPL * E;

  const int lane = threadIdx.x & (kWave - 1);
  const int64_t wave = int64_t(blockIdx.x) * (blockDim.x / kWave) + wave_in_block();
  const int64_t base = wave * TILE;
  if (base >= n) return;

  if (vec_ok && base + TILE <= n) {
    const int64_t vbase = base / E;
    const int64_t wbase = base / 16;
    u32x4 in[VPL];
    uint32_t part[VPL];
#pragma unroll
    for (int j = 0; j < VPL; ++j) in[j] = ldg16<kActNtLoad>(dy, vbase + j * kWave + lane);
    load_tile_codes<IO, VPL>(codes, wbase, part, lane);
#pragma unroll
    for (int j = 0; j < VPL; ++j) {
      const uint32_t p = part[j];
      float f[E];
      IO::unpack(in[j], f);
#pragma unroll
      for (int e = 0; e < E; ++e) f[e] = f[e] * seg_slope<A>((p >> (2 * e)) & 3u);
      stb16<LMBP_ACT_STORE_CPOL>(vec_rsrc(dx, vbase, VPL * kWave), j * kWave + lane, IO::pack(f));
    }
    return;
  }

  const int64_t end = (base + TILE < n) ? base + TILE : n;
  for (int64_t i = base + lane; i < end; i += kWave) {
    const uint32_t c = (codes[i / 16] >> (2 * (i % 16))) & 3u;
    IO::store1(dx, i, IO::load1(dy, i) * seg_slope<A>(c));
  }
}

// ReSiLU2 (or ReGELU2) inside a gated product h = act(g) * u (SwiGLU when act is
// SiLU). Forward writes h, s = act(g) (what the product's backward needs) and the
// codes of g; backward: dg = dh * u * slope[code], du = dh * s. Same tiling as the
// plain activation kernels; fusing saves the round trip of s and ds through HBM.
template <class IO, int ACT, int VPL>
__global__ __launch_bounds__(LMBP_ACT_BLOCK) void glu_fwd_kernel(const void* g, const void* u, void* h,
                                                                 void* s, uint32_t* __restrict__ codes,
                                                                 int64_t n, int vec_ok) {
  using A = ActOf<ACT>;
  constexpr bool kPrecise = std::is_same<IO, F32>::value;
  constexpr int E = IO::kPerVec;
  constexpr int TILE = kWave * VPL * E;
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t wave = int64_t(blockIdx.x) * (blockDim.x / kWave) + wave_in_block();
  const int64_t base = wave * TILE;
  if (base >= n) return;

  if (vec_ok && base + TILE <= n) {
    const int64_t vbase = base / E;
    u32x4 vg[VPL], vu[VPL];
#pragma unroll
    for (int j = 0; j < VPL; ++j) {
      vg[j] = ldg16<kActNtLoad>(g, vbase + j * kWave + lane);
      vu[j] = ldg16<kActNtLoad>(u, vbase + j * kWave + lane);
    }
    uint32_t part[VPL];
#pragma unroll
    for (int j = 0; j < VPL; ++j) {
      float fg[E], fu[E], fs[E];
      IO::unpack(vg[j], fg);
      IO::unpack(vu[j], fu);
#pragma unroll
      for (int e = 0; e < E; ++e) gated_value<ACT, kPrecise>(fg[e], fu[e], fs[e], fu[e]);
      part[j] = codes_of<A>(fg);
      stb16<LMBP_GLU_STORE_CPOL>(vec_rsrc(s, vbase, VPL * kWave), j * kWave + lane, IO::pack(fs));
      stb16<LMBP_GLU_STORE_CPOL>(vec_rsrc(h, vbase, VPL * kWave), j * kWave + lane, IO::pack(fu));
    }
    store_tile_codes<IO, VPL>(codes, base / 16, part, lane);
    return;
  }

  const int64_t end = (base + TILE < n) ? base + TILE : n;
  const int64_t w_end = (end + 15) / 16;
  for (int64_t w = base / 16 + lane; w < w_end; w += kWave) {
    uint32_t word = 0;
    for (int e = 0; e < 16; ++e) {
      const int64_t i = w * 16 + e;
      if (i < n) {
        const float gv = IO::load1(g, i);
        const float uv = IO::load1(u, i);
        float sv, hv;
        gated_value<ACT, kPrecise>(gv, uv, sv, hv);
        IO::store1(s, i, sv);
        IO::store1(h, i, hv);
        word |= seg_code<A>(gv) << (2 * e);
      }
    }
    codes[w] = word;
  }
}

template <class IO, int ACT, int VPL>
__global__ __launch_bounds__(LMBP_ACT_BLOCK) void glu_bwd_kernel(const void* dh, const void* u,
                                                                 const void* s,
                                                                 const uint32_t* __restrict__ codes,
                                                                 void* dg, void* du, int64_t n,
                                                                 int vec_ok) {
  using A = ActOf<ACT>;
  constexpr int E = IO::kPerVec;
  constexpr int TILE = kWave * VPL * E;
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t wave = int64_t(blockIdx.x) * (blockDim.x / kWave) + wave_in_block();
  const int64_t base = wave * TILE;
  if (base >= n) return;

  if (vec_ok && base + TILE <= n) {
    const int64_t vbase = base / E;
    u32x4 vh[VPL], vu[VPL], vs[VPL];
    uint32_t part[VPL];
#pragma unroll
    for (int j = 0; j < VPL; ++j) {
      vh[j] = ldg16<kActNtLoad>(dh, vbase + j * kWave + lane);
      vu[j] = ldg16<kActNtLoad>(u, vbase + j * kWave + lane);
      vs[j] = ldg16<kActNtLoad>(s, vbase + j * kWave + lane);
    }
    load_tile_codes<IO, VPL>(codes, base / 16, part, lane);
#pragma unroll
    for (int j = 0; j < VPL; ++j) {
      float fh[E], fu[E], fs[E];
      IO::unpack(vh[j], fh);
      IO::unpack(vu[j], fu);
      IO::unpack(vs[j], fs);
#pragma unroll
      for (int e = 0; e < E; ++e) {
        fu[e] = fh[e] * fu[e] * seg_slope<A>((part[j] >> (2 * e)) & 3u);   // dg
        fs[e] = fh[e] * fs[e];                                              // du
      }
      stb16<LMBP_GLU_STORE_CPOL>(vec_rsrc(dg, vbase, VPL * kWave), j * kWave + lane, IO::pack(fu));
      stb16<LMBP_GLU_STORE_CPOL>(vec_rsrc(du, vbase, VPL * kWave), j * kWave + lane, IO::pack(fs));
    }
    return;
  }

  const int64_t end = (base + TILE < n) ? base + TILE : n;
  for (int64_t i = base + lane; i < end; i += kWave) {
    const uint32_t c = (codes[i / 16] >> (2 * (i % 16))) & 3u;
    const float hv = IO::load1(dh, i);
    const float uv = IO::load1(u, i);
    const float sv = IO::load1(s, i);
    IO::store1(dg, i, hv * uv * seg_slope<A>(c));
    IO::store1(du, i, hv * sv);
  }
}

// ------------------------------------------------------------------ launchers
namespace {
template <class IO, int V>
constexpr int fit_vpl() {
  // 1, or a multiple of the lanes sharing a code word (2 for bf16, 4 for fp32).
  constexpr int g = 16 / IO::kPerVec;
  return (V == 1 || V % g == 0) ? V : ((V + g - 1) / g) * g;
}
template <class IO>
constexpr int act_vpl() {
  return std::is_same<IO, F32>::value ? fit_vpl<IO, LMBP_ACT_VPL_F32>() : fit_vpl<IO, LMBP_ACT_VPL>();
}
template <class IO>
constexpr int glu_vpl() {
  return std::is_same<IO, BF16>::value ? fit_vpl<IO, LMBP_GLU_VPL>() : act_vpl<IO>();
}
template <class IO>
constexpr int act_block() { return std::is_same<IO, F32>::value ? LMBP_ACT_BLOCK_F32 : LMBP_ACT_BLOCK; }
template <class IO, int VPL>
int64_t tile_blocks(int64_t n) {
  constexpr int wpb = act_block<IO>() / kWave;
  constexpr int64_t tile = int64_t(kWave) * VPL * IO::kPerVec;
  const int64_t waves = (n + tile - 1) / tile;
  return (waves + wpb - 1) / wpb;
}
template <class IO>
int64_t act_blocks(int64_t n) { return tile_blocks<IO, act_vpl<IO>()>(n); }
template <class IO>
int64_t glu_blocks(int64_t n) { return tile_blocks<IO, glu_vpl<IO>()>(n); }
}  // namespace

template <class IO, int ACT>
hipError_t launch_act_fwd_t(int64_t n, const void* x, void* y, uint32_t* codes, bool vec_ok,
                            hipStream_t s) {
  const int64_t blocks = act_blocks<IO>(n);
  if (blocks > 0x7fffffff) return hipErrorInvalidValue;
  hipLaunchKernelGGL((act_fwd_kernel<IO, ACT, act_vpl<IO>()>), dim3(unsigned(blocks)), dim3(act_block<IO>()), 0, s,
                     x, y, codes, n, int(vec_ok));
  return hipGetLastError();
}

template <class IO, int ACT>
hipError_t launch_act_bwd_t(int64_t n, const void* dy, const uint32_t* codes, void* dx,
                            bool vec_ok, hipStream_t s) {
  const int64_t blocks = act_blocks<IO>(n);
  if (blocks > 0x7fffffff) return hipErrorInvalidValue;
  hipLaunchKernelGGL((act_bwd_kernel<IO, ACT, act_vpl<IO>()>), dim3(unsigned(blocks)), dim3(act_block<IO>()), 0, s,
                     dy, codes, dx, n, int(vec_ok));
  return hipGetLastError();
}

template <class IO, int ACT>
hipError_t launch_glu_fwd_t(int64_t n, const void* g, const void* u, void* h, void* s,
                            uint32_t* codes, bool vec_ok, hipStream_t st) {
  const int64_t blocks = glu_blocks<IO>(n);
  if (blocks > 0x7fffffff) return hipErrorInvalidValue;
  hipLaunchKernelGGL((glu_fwd_kernel<IO, ACT, glu_vpl<IO>()>), dim3(unsigned(blocks)),
                     dim3(act_block<IO>()), 0, st, g, u, h, s, codes, n, int(vec_ok));
  return hipGetLastError();
}

template <class IO, int ACT>
hipError_t launch_glu_bwd_t(int64_t n, const void* dh, const void* u, const void* s,
                            const uint32_t* codes, void* dg, void* du, bool vec_ok, hipStream_t st) {
  const int64_t blocks = glu_blocks<IO>(n);
  if (blocks > 0x7fffffff) return hipErrorInvalidValue;
  hipLaunchKernelGGL((glu_bwd_kernel<IO, ACT, glu_vpl<IO>()>), dim3(unsigned(blocks)),
                     dim3(act_block<IO>()), 0, st, dh, u, s, codes, dg, du, n, int(vec_ok));
  return hipGetLastError();
}

hipError_t launch_glu_fwd(int act, bool bf16, int64_t n, const void* g, const void* u, void* h,
                          void* s, uint32_t* codes, bool vec_ok, hipStream_t st) {
  if (act != kSilu) return hipErrorInvalidValue;
  return bf16 ? launch_glu_fwd_t<BF16, kSilu>(n, g, u, h, s, codes, vec_ok, st)
              : launch_glu_fwd_t<F32, kSilu>(n, g, u, h, s, codes, vec_ok, st);
}

hipError_t launch_glu_bwd(int act, bool bf16, int64_t n, const void* dh, const void* u,
                          const void* s, const uint32_t* codes, void* dg, void* du, bool vec_ok,
                          hipStream_t st) {
  if (act != kSilu) return hipErrorInvalidValue;
  return bf16 ? launch_glu_bwd_t<BF16, kSilu>(n, dh, u, s, codes, dg, du, vec_ok, st)
              : launch_glu_bwd_t<F32, kSilu>(n, dh, u, s, codes, dg, du, vec_ok, st);
}

hipError_t launch_act_fwd(int act, bool bf16, int64_t n, const void* x, void* y,
                          uint32_t* codes, bool vec_ok, hipStream_t s) {
  if (act == kGelu)
    return bf16 ? launch_act_fwd_t<BF16, kGelu>(n, x, y, codes, vec_ok, s)
                : launch_act_fwd_t<F32, kGelu>(n, x, y, codes, vec_ok, s);
  return bf16 ? launch_act_fwd_t<BF16, kSilu>(n, x, y, codes, vec_ok, s)
              : launch_act_fwd_t<F32, kSilu>(n, x, y, codes, vec_ok, s);
}

hipError_t launch_act_bwd(int act, bool bf16, int64_t n, const void* dy, const uint32_t* codes,
                          void* dx, bool vec_ok, hipStream_t s) {
  if (act == kGelu)
    return bf16 ? launch_act_bwd_t<BF16, kGelu>(n, dy, codes, dx, vec_ok, s)
                : launch_act_bwd_t<F32, kGelu>(n, dy, codes, dx, vec_ok, s);
  return bf16 ? launch_act_bwd_t<BF16, kSilu>(n, dy, codes, dx, vec_ok, s)
              : launch_act_bwd_t<F32, kSilu>(n, dy, codes, dx, vec_ok, s);
}

}  // namespace lmbp
