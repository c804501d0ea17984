// Exact GELU and SiLU in fp32 for the activation kernels (gfx950).
#pragma once

#include "gelu_poly.h"
#include "lmbp_device.hpp"
#include "lmbp_launch.hpp"

namespace lmbp {

// ------------------------------------------------------------- activations
// exp2 on the hardware unit (v_exp_f32); arguments here are never NaN.
__device__ inline float hw_exp2(float v) { return __builtin_amdgcn_exp2f(v); }
__device__ inline float hw_rcp(float v) { return __builtin_amdgcn_rcpf(v); }
// max(x, 0) as one v_max_f32. The compiler's fmaxf first quiets a possible
// signalling NaN with an extra max of x with itself (IEEE mode); inputs here are
// finite, so that operation is pure overhead.
__device__ inline float hw_relu(float x) {
  float r;
  asm("v_max_f32 %0, 0, %1" : "=v"(r) : "v"(x));
  return r;
}
// min(t, hi) for t >= 0 as one v_med3_f32 (median of t, hi and 0), likewise
// without the quieting operation of fminf.
__device__ inline float hw_clamp_hi(float t, float hi) { return __builtin_amdgcn_fmed3f(t, hi, 0.0f); }

// GELU(x) = x Phi(x). With t = |x| and Q(t) = 1 - Phi(t): Phi(x) = Q(t) for x < 0 and
// 1 - Q(t) otherwise, so GELU(x) = max(x, 0) - t Q(t) for either sign (one fused
// multiply-add, rounded once). The polynomials come from gelu_poly.h; their domain ends
// at T = 13.5, beyond which t Q(t) < 2^-126 and the result is max(x, 0) up to a
// subnormal.
//   PRECISE (fp32 storage): Q(t) = 2^E, E = -(log2 e / 2) t^2 + R(v), R of degree 14 in
//   v = min(t, T) (2/T) - 1. The quadratic term is carried in two pieces and the
//   exponent split into integer and fraction, so that no rounding of the large exponent
//   reaches the result; ldexp forms subnormal Q exactly (relative error below 1e-6).
//   Otherwise (bf16 storage): u = min(t / T, 1) in one multiply whose result the
//   hardware clamps to [0, 1], then t Q(t) = u 2^P(u) with P of degree 8 (the quadratic
//   folded in). 2^P(u) >= t Q(t) >= 2^-126 wherever the result is a normal number, so
//   the exponential unit's flushing of subnormal results never drops one.
constexpr double kLog2eHalf = 0.72134752044448170368;  // log2(e) / 2
constexpr float kLog2eHalfHi = static_cast<float>(kLog2eHalf);
constexpr float kLog2eHalfLo = static_cast<float>(kLog2eHalf - static_cast<double>(kLog2eHalfHi));

template <int D>
__device__ inline float horner(const float (&c)[D], float v) {
  float r = c[0];
#pragma unroll
  for (int k = 1; k < D; ++k) r = __builtin_fmaf(r, v, c[k]);
  return r;
}

// min(|x| * s, 1) for s > 0: one v_mul_f32 with the clamp output modifier (results
// clamped to [0, 1]; the product is never NaN for finite x).
__device__ inline float abs_mul_clamp01(float x, float s) {
  float r;
  asm("v_mul_f32_e64 %0, |%1|, %2 clamp" : "=v"(r) : "v"(x), "v"(s));
  return r;
}

template <bool PRECISE>
__device__ inline float gelu_f(float x) {
  if constexpr (PRECISE) {
    const float t = __builtin_fabsf(x);
    const float v = __builtin_fmaf(hw_clamp_hi(t, LMBP_GELU_T), LMBP_GELU_2_OVER_T, -1.0f);
    const float r = horner(kGeluR14, v);
    const float tc = hw_clamp_hi(t, 16.0f);   // Q is 0 in fp32 beyond: keeps E finite
    const float a_hi = tc * -kLog2eHalfHi;
    const float a_lo = __builtin_fmaf(tc, -kLog2eHalfLo, __builtin_fmaf(tc, -kLog2eHalfHi, -a_hi));
    const float k = __builtin_rintf(__builtin_fmaf(tc, a_hi, r));
    const float f = __builtin_fmaf(tc, a_hi, -k) + __builtin_fmaf(tc, a_lo, r);
    const float q = __builtin_ldexpf(hw_exp2(f), int(k));
    return __builtin_fmaf(-t, q, hw_relu(x));
  } else {
    const float u = abs_mul_clamp01(x, LMBP_GELU_INV_T);
    const float q = hw_exp2(horner(kGeluP8, u));
    return __builtin_fmaf(-u, q, hw_relu(x));
  }
}

// SiLU(x) = x / (1 + e^-x), with the exponential taken with a bias so that no
// intermediate overflows and none that matters is flushed (the plain form x rcp(1 + e^-x)
// overflowed below x = -88.7 and returned -0 where the true value, e.g. -2e-37 at
// x = -89, is a normal number).
//   bf16 storage: e = 2^(-x log2 e - 16) = e^-x 2^-16 (finite down to x = -99.8) and
//   r = 1 / (2^-16 + e) = 2^16 sigmoid(x), a normal number down to x = -98.4.
//   SiLU(x) = x (r 2^-16): the factor is the sigmoid itself, subnormal below x = -87.3
//   (at least 16 significant bits while the result is normal, down to -91.9).
//   PRECISE (fp32 storage): with t = |x| and e_s = e^-t 2^8 (normal for t <= 92.9),
//   x sigmoid(x) = max(x, 0) - t e^-t / (1 + e^-t) = max(x, 0) - (t e_s) / (2^8 + e_s):
//   no intermediate is subnormal while the result is normal. The exponent is split into
//   integer k and fraction f, the rounding error of t log2 e carried into f and 2^(8-k)
//   applied with ldexp, so the exponent's rounding does not reach the result.
constexpr double kLog2e = 1.44269504088896340736;
constexpr float kLog2eHi = static_cast<float>(kLog2e);
constexpr float kLog2eLo = static_cast<float>(kLog2e - static_cast<double>(kLog2eHi));

// 2^16 sigmoid(x) (bf16-storage form).
__device__ inline float sigmoid_x64k(float x) {
  return hw_rcp(hw_exp2(__builtin_fmaf(x, -kLog2eHi, -16.0f)) + 0x1p-16f);
}

template <bool PRECISE>
__device__ inline float silu_f(float x) {
  if constexpr (PRECISE) {
    const float t = __builtin_fabsf(x);
    const float tc = hw_clamp_hi(t, 128.0f);   // e_s is 0 beyond: keeps p finite
    const float p = tc * kLog2eHi;
    const float p_lo = __builtin_fmaf(tc, kLog2eLo, __builtin_fmaf(tc, kLog2eHi, -p));
    const float k = __builtin_rintf(p);
    const float e_s = __builtin_ldexpf(hw_exp2((k - p) - p_lo), 8 - int(k));
    return __builtin_fmaf(-(t * e_s), hw_rcp(e_s + 256.0f), hw_relu(x));
  } else {
    return x * (sigmoid_x64k(x) * 0x1p-16f);
  }
}

template <int ACT, bool PRECISE>
__device__ inline float act_value(float x) {
  if constexpr (ACT == kGelu) return gelu_f<PRECISE>(x);
  else return silu_f<PRECISE>(x);
}

// Gated product h = act(g) u together with s = act(g) (SwiGLU when act is SiLU). For SiLU
// with bf16 storage the product is formed from the scaled value g r = 2^16 SiLU(g), a
// normal number while SiLU(g) >= 2^-142, and only then scaled back: h keeps full precision
// where SiLU(g) itself is subnormal but h is not (g near -93 with |u| > 3, say). That form
// needs |g| < 2^112 (above, g r overflows); fp32 storage and GELU use s u directly.
template <int ACT, bool PRECISE>
__device__ inline void gated_value(float g, float u, float& s, float& h) {
  if constexpr (ACT == kSilu && !PRECISE) {
    const float gr = g * sigmoid_x64k(g);
    s = gr * 0x1p-16f;
    h = (gr * u) * 0x1p-16f;
  } else {
    s = act_value<ACT, PRECISE>(g);
    h = s * u;
  }
}

}  // namespace lmbp
