// Constants of the three-ReLU combinations (Appendix E) and the 2-bit segment
// codes of ReGELU2 / ReSiLU2 (Sec. 4.2, eq. relus_family with k = 2), shared by the
// activation kernels and the fused linear-layer epilogue.
#pragma once

#include "lmbp_device.hpp"
#include "lmbp_launch.hpp"

#include <type_traits>

namespace lmbp {

// ------------------------------------------------------------------ constants
// Appendix E: weights a* and biases c* of the three-ReLU combinations.
struct GeluConsts {
  static constexpr double a1 = -0.04922261145617846;
  static constexpr double a2 = 1.0979632065417297;
  static constexpr double c1 = -3.1858810036855245;
  static constexpr double c2 = -0.001178821281161997;
  static constexpr double c3 = 3.190832613414926;
};
struct SiluConsts {
  static constexpr double a1 = -0.04060357190528599;
  static constexpr double a2 = 1.080925428529668;
  static constexpr double c1 = -6.3050461001646445;
  static constexpr double c2 = -0.0008684942046214787;
  static constexpr double c3 = 6.325815242089708;
};

constexpr float f32_step(float f, int dir) {  // one ulp toward +inf (dir>0) or -inf
  uint32_t b = __builtin_bit_cast(uint32_t, f);
  const bool neg = (b >> 31) != 0u;
  b = ((dir > 0) != neg) ? b + 1u : b - 1u;
  return __builtin_bit_cast(float, b);
}
constexpr float round_down_f32(double c) {
  const float f = static_cast<float>(c);
  return (static_cast<double>(f) > c) ? f32_step(f, -1) : f;
}

// The code compares in fp32: for any fp32 (or bf16) value x and a bias c that is
// not representable in fp32, x > c holds exactly when x > RD(c), RD(c) being the
// largest fp32 value below c. The static_asserts check non-representability, so
// the comparison is exact and no tie rule is ever needed.
template <class C>
struct Act {
  static constexpr float t1 = round_down_f32(C::c1);
  static constexpr float t2 = round_down_f32(C::c2);
  static constexpr float t3 = round_down_f32(C::c3);
  static_assert(static_cast<double>(t1) < C::c1 && C::c1 < static_cast<double>(f32_step(t1, 1)), "c1");
  static_assert(static_cast<double>(t2) < C::c2 && C::c2 < static_cast<double>(f32_step(t2, 1)), "c2");
  static_assert(static_cast<double>(t3) < C::c3 && C::c3 < static_cast<double>(f32_step(t3, 1)), "c3");
  // Slopes of the combination on segments 1 and 2 (segment 0: 0, segment 3: 1).
  static constexpr float s1 = static_cast<float>(C::a1);
  static constexpr float s2 = static_cast<float>(C::a1 + C::a2);
};
using GeluAct = Act<GeluConsts>;
using SiluAct = Act<SiluConsts>;

template <class A>
__device__ inline uint32_t seg_code(float x) {
  // code = [x > c1] + [x > c2] + [x > c3] for c1 < c2 < c3, written as its two bits:
  // bit 1 = [x > c2], bit 0 = [x > c1] xor [x > c2] xor [x > c3].
  const uint32_t b1 = x > A::t2;
  const uint32_t b0 = uint32_t(x > A::t1) ^ b1 ^ uint32_t(x > A::t3);
  return b0 | (b1 << 1);
}

#ifndef LMBP_ACT_CARRY_CODES
#define LMBP_ACT_CARRY_CODES 1  // vector-path codes through compare masks and carry-in adds
#endif

// Codes of E elements, element e in bits 2e (bit 0 of its code) and 2e + 1 (bit 1),
// built without materialising any per-element bool: each compare leaves a lane
// mask, bit 0's masks are combined with scalar xors, and each bit enters the word
// as the carry input of an add of the word to itself (p = 2p + bit, last element
// first). That is three compares and two adds per element, against about eight
// vector operations for the select-and-shift form.
__device__ inline uint32_t shift_in(uint32_t p, uint64_t lane_mask) {
  uint32_t r;
  uint64_t carry_out;
  asm("v_addc_co_u32_e64 %0, %1, %2, %2, %3" : "=v"(r), "=s"(carry_out) : "v"(p), "s"(lane_mask));
  return r;
}

template <class A, int E>
__device__ inline uint32_t codes_of(const float (&f)[E]) {
  uint32_t p = 0;
#if LMBP_ACT_CARRY_CODES
#pragma unroll
  for (int e = E - 1; e >= 0; --e) {
    const uint64_t m2 = __builtin_amdgcn_ballot_w64(f[e] > A::t2);
    const uint64_t m0 = __builtin_amdgcn_ballot_w64(f[e] > A::t1) ^ m2 ^
                        __builtin_amdgcn_ballot_w64(f[e] > A::t3);
    p = shift_in(shift_in(p, m2), m0);
  }
#else
#pragma unroll
  for (int e = 0; e < E; ++e) p |= seg_code<A>(f[e]) << (2 * e);
#endif
  return p;
}

template <class A>
__device__ inline float seg_slope(uint32_t c) {
  return (c & 2u) ? ((c & 1u) ? 1.0f : A::s2) : ((c & 1u) ? A::s1 : 0.0f);
}

template <int ACT>
using ActOf = typename std::conditional<ACT == kGelu, GeluAct, SiluAct>::type;

}  // namespace lmbp
