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

// GELU(x) = x Phi(x). With t = |x| and Q(t) = 1 - Phi(t) = 2^E(t),
// E(t) = -(log2 e / 2) t^2 + R(t), where R is the fitted polynomial of
// gelu_poly.h (argument clamped to [0, T]). Phi(x) = Q(t) for x < 0 and 1 - Q(t)
// otherwise, so GELU(x) = max(x, 0) - t Q(t) for either sign: one fused
// multiply-add (rounded once) instead of a select, a subtraction and a product.
//   PRECISE (fp32 storage): degree-12 R; the quadratic term is carried in two
//   pieces and the exponent split into integer and fraction so that no rounding
//   of the large exponent reaches the result (relative error below 1e-6).
//   Otherwise (bf16 storage): degree-8 R, single-piece exponent (about 1e-5).
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

template <bool PRECISE>
__device__ inline float gelu_f(float x) {
  const float t = __builtin_fabsf(x);
  const float v = __builtin_fmaf(hw_clamp_hi(t, LMBP_GELU_T), LMBP_GELU_2_OVER_T, -1.0f);
  float q;
  if constexpr (PRECISE) {
    const float r = horner(kGeluR12, v);
    const float a_hi = t * -kLog2eHalfHi;
    const float a_lo = __builtin_fmaf(t, -kLog2eHalfLo, __builtin_fmaf(t, -kLog2eHalfHi, -a_hi));
    const float e0 = __builtin_fmaxf(__builtin_fmaf(t, a_hi, r), -256.0f);
    const float k = __builtin_rintf(e0);
    const float f = __builtin_fmaf(t, a_hi, -k) + __builtin_fmaf(t, a_lo, r);
    q = __builtin_ldexpf(hw_exp2(f), int(k));
  } else {
    const float r = horner(kGeluR8, v);
    q = hw_exp2(__builtin_fmaf(t, t * -kLog2eHalfHi, r));
  }
  return __builtin_fmaf(-t, q, hw_relu(x));
}

// SiLU(x) = x / (1 + 2^(-x log2 e)).
//   PRECISE: the exponent's rounding error is carried separately and applied as a
//   first-order factor (1 + err ln 2) (product form, so an infinite 2^a stays inf).
constexpr double kLog2e = 1.44269504088896340736;
constexpr float kLog2eHi = static_cast<float>(kLog2e);
constexpr float kLog2eLo = static_cast<float>(kLog2e - static_cast<double>(kLog2eHi));
constexpr float kLn2 = 0.69314718055994530942f;

template <bool PRECISE>
__device__ inline float silu_f(float x) {
  const float a = x * -kLog2eHi;
  float e = hw_exp2(a);
  if constexpr (PRECISE) {
    const float a_lo = __builtin_fmaf(x, -kLog2eLo, __builtin_fmaf(x, -kLog2eHi, -a));
    e = e * __builtin_fmaf(a_lo, kLn2, 1.0f);
  }
  return x * hw_rcp(1.0f + e);
}

template <int ACT, bool PRECISE>
__device__ inline float act_value(float x) {
  if constexpr (ACT == kGelu) return gelu_f<PRECISE>(x);
  else return silu_f<PRECISE>(x);
}

}  // namespace lmbp
