// Device-side building blocks shared by the lmbp kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lmbp {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;

// Storage formats. A "vector" is 16 bytes: 4 fp32 or 8 bf16 elements.
struct F32 {
  static constexpr int kBytes = 4;
  static constexpr int kPerVec = 4;
  static __device__ inline float load1(const void* p, int64_t i) {
    return reinterpret_cast<const float*>(p)[i];
  }
  static __device__ inline void store1(void* p, int64_t i, float v) {
    reinterpret_cast<float*>(p)[i] = v;
  }
  // Decode the 4 elements of a vector.
  static __device__ inline void unpack(const u32x4& v, float (&f)[4]) {
#pragma unroll
    for (int k = 0; k < 4; ++k) f[k] = __uint_as_float(v[k]);
  }
  static __device__ inline u32x4 pack(const float (&f)[4]) {
    u32x4 v;
#pragma unroll
    for (int k = 0; k < 4; ++k) v[k] = __float_as_uint(f[k]);
    return v;
  }
};

// bf16 -> fp32 is exact (append 16 zero bits); fp32 -> bf16 rounds to nearest
// even with the gfx950 packed conversion (v_cvt_pk_bf16_f32).
__device__ inline uint32_t pack_bf16x2(float lo, float hi) {
  f32x2 f = {lo, hi};
  bf16x2 h = __builtin_convertvector(f, bf16x2);
  return __builtin_bit_cast(uint32_t, h);
}

struct BF16 {
  static constexpr int kBytes = 2;
  static constexpr int kPerVec = 8;
  static __device__ inline float load1(const void* p, int64_t i) {
    return __uint_as_float(uint32_t(reinterpret_cast<const uint16_t*>(p)[i]) << 16);
  }
  static __device__ inline void store1(void* p, int64_t i, float v) {
    reinterpret_cast<uint16_t*>(p)[i] = uint16_t(pack_bf16x2(v, 0.0f) & 0xffffu);
  }
  static __device__ inline void unpack(const u32x4& v, float (&f)[8]) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      f[2 * k] = __uint_as_float(v[k] << 16);
      f[2 * k + 1] = __uint_as_float(v[k] & 0xffff0000u);
    }
  }
  static __device__ inline u32x4 pack(const float (&f)[8]) {
    u32x4 v;
#pragma unroll
    for (int k = 0; k < 4; ++k) v[k] = pack_bf16x2(f[2 * k], f[2 * k + 1]);
    return v;
  }
};

// 16-byte global loads / stores. NT selects the non-temporal (streaming) cache
// policy, for data that is touched exactly once.
template <bool NT = false>
__device__ inline u32x4 ldg16(const void* base, int64_t vec_index) {
  const u32x4* p = reinterpret_cast<const u32x4*>(base) + vec_index;
  if constexpr (NT) return __builtin_nontemporal_load(p);
  else return *p;
}
template <bool NT = false>
__device__ inline void stg16(void* base, int64_t vec_index, const u32x4& v) {
  u32x4* p = reinterpret_cast<u32x4*>(base) + vec_index;
  if constexpr (NT) __builtin_nontemporal_store(v, p);
  else *p = v;
}

// Wave index within the block as a wave-uniform (scalar) value.
__device__ inline int wave_in_block() {
  return __builtin_amdgcn_readfirstlane(int(threadIdx.x) / kWave);
}

// Buffer resource over the 16-byte vectors [vbase, vbase + nvec) of `base` (both
// wave-uniform), and a 16-byte store through it with cache policy CPOL (buffer
// instruction bits: sc0 = 1, nt = 2, sc1 = 16).
__device__ inline __amdgpu_buffer_rsrc_t vec_rsrc(void* base, int64_t vbase, int64_t nvec) {
  return __builtin_amdgcn_make_buffer_rsrc(static_cast<char*>(base) + vbase * 16, 0, int(nvec * 16),
                                           0x00020000);
}
template <int CPOL = 2 | 16>
__device__ inline void stb16(__amdgpu_buffer_rsrc_t r, int idx, const u32x4& v) {
  __builtin_amdgcn_raw_buffer_store_b128(v, r, idx * 16, 0, CPOL);
}

// Compiler-only barrier: makes `v` opaque so that values derived from it are
// recomputed after this point instead of being kept live in registers.
__device__ inline void opaque(u32x4& v) { asm volatile("" : "+v"(v)); }

// Cross-lane move inside groups of 4 lanes (DPP quad_perm): lane q of every quad
// receives `v` from lane perm[q] of the same quad.
template <int P0, int P1, int P2, int P3>
__device__ inline uint32_t quad_perm(uint32_t v) {
  constexpr int ctrl = P0 | (P1 << 2) | (P2 << 4) | (P3 << 6);
  return uint32_t(__builtin_amdgcn_update_dpp(0, int(v), ctrl, 0xf, 0xf, false));
}

// Lane q of each group of G lanes (G = 2 or 4) receives v from lane (q + S) mod G.
template <int G, int S>
__device__ inline uint32_t group_rotate(uint32_t v) {
  static_assert(G == 2 || G == 4, "group size");
  if constexpr (S % G == 0) {
    return v;
  } else if constexpr (G == 2) {
    return quad_perm<1, 0, 3, 2>(v);
  } else {
    return quad_perm<(0 + S) % 4, (1 + S) % 4, (2 + S) % 4, (3 + S) % 4>(v);
  }
}

__device__ inline float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, kWave);
  return v;
}

// Sum of `v` over the block (blockDim.x a multiple of 64, at most 1024 threads);
// every thread gets the total. `scratch` holds at least blockDim.x / 64 floats.
__device__ inline float block_sum(float v, float* scratch) {
  const int lane = threadIdx.x & (kWave - 1);
  const int wid = threadIdx.x / kWave;
  const int nw = blockDim.x / kWave;
  v = wave_sum(v);
  __syncthreads();  // scratch may still be read by a previous reduction
  if (lane == 0) scratch[wid] = v;
  __syncthreads();
  float t = 0.0f;
  for (int w = 0; w < nw; ++w) t += scratch[w];  // same order in every thread
  return t;
}

}  // namespace lmbp
