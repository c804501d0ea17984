// C ABI of liblmbp (declared in include/lmbp.h): host-side validation, path
// selection and launch. Nothing here allocates, frees or synchronizes.
#include "lmbp.h"
#include "lmbp_launch.hpp"

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <limits>

namespace {

thread_local int g_last_hip_error = 0;

struct Span {
  uintptr_t lo, hi;  // [lo, hi)
};

Span span(const void* p, uint64_t bytes) {
  const uintptr_t a = reinterpret_cast<uintptr_t>(p);
  return Span{a, a + bytes};
}

bool overlaps(Span a, Span b) {
  return a.lo < b.hi && b.lo < a.hi && a.hi > a.lo && b.hi > b.lo;
}

// Two buffers of a call may either be disjoint or, when `same_ok`, identical.
bool bad_pair(Span a, Span b, bool same_ok) {
  if (!overlaps(a, b)) return false;
  return !(same_ok && a.lo == b.lo && a.hi == b.hi);
}

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

int elem_bytes(lmbp_dtype dt) { return dt == LMBP_BF16 ? 2 : 4; }

bool known_dtype(int dt) { return dt == LMBP_FP32 || dt == LMBP_BF16; }

lmbp_status from_hip(hipError_t e) {
  if (e == hipSuccess) return LMBP_OK;
  g_last_hip_error = int(e);
  return LMBP_EHIP;
}

lmbp_status act_fwd(int act, lmbp_dtype dt, int64_t n, const void* x, void* y, uint32_t* codes,
                    void* stream) {
  if (!known_dtype(dt)) return LMBP_EDTYPE;
  if (n < 0 || uint64_t(n) > (uint64_t(1) << 60)) return LMBP_EINVAL;
  if (n == 0) return LMBP_OK;
  if (!x || !y || !codes) return LMBP_EINVAL;
  const int eb = elem_bytes(dt);
  if (!aligned(x, eb) || !aligned(y, eb) || !aligned(codes, 4)) return LMBP_EINVAL;
  const Span sx = span(x, uint64_t(n) * eb), sy = span(y, uint64_t(n) * eb);
  const Span sc = span(codes, lmbp_codes_bytes(n));
  if (bad_pair(sx, sy, true) || bad_pair(sc, sx, false) || bad_pair(sc, sy, false))
    return LMBP_EOVERLAP;
  const bool vec_ok = aligned(x, 16) && aligned(y, 16);
  return from_hip(lmbp::launch_act_fwd(act, dt == LMBP_BF16, n, x, y, codes, vec_ok,
                                       static_cast<hipStream_t>(stream)));
}

lmbp_status act_bwd(int act, lmbp_dtype dt, int64_t n, const void* dy, const uint32_t* codes,
                    void* dx, void* stream) {
  if (!known_dtype(dt)) return LMBP_EDTYPE;
  if (n < 0 || uint64_t(n) > (uint64_t(1) << 60)) return LMBP_EINVAL;
  if (n == 0) return LMBP_OK;
  if (!dy || !dx || !codes) return LMBP_EINVAL;
  const int eb = elem_bytes(dt);
  if (!aligned(dy, eb) || !aligned(dx, eb) || !aligned(codes, 4)) return LMBP_EINVAL;
  const Span sg = span(dy, uint64_t(n) * eb), sd = span(dx, uint64_t(n) * eb);
  const Span sc = span(codes, lmbp_codes_bytes(n));
  if (bad_pair(sg, sd, true) || bad_pair(sc, sg, false) || bad_pair(sc, sd, false))
    return LMBP_EOVERLAP;
  const bool vec_ok = aligned(dy, 16) && aligned(dx, 16);
  return from_hip(lmbp::launch_act_bwd(act, dt == LMBP_BF16, n, dy, codes, dx, vec_ok,
                                       static_cast<hipStream_t>(stream)));
}

lmbp_status glu_fwd(lmbp_dtype dt, int64_t n, const void* g, const void* u, void* h, void* s,
                    uint32_t* codes, void* stream) {
  if (!known_dtype(dt)) return LMBP_EDTYPE;
  if (n < 0 || uint64_t(n) > (uint64_t(1) << 60)) return LMBP_EINVAL;
  if (n == 0) return LMBP_OK;
  if (!g || !u || !h || !s || !codes) return LMBP_EINVAL;
  const int eb = elem_bytes(dt);
  if (!aligned(g, eb) || !aligned(u, eb) || !aligned(h, eb) || !aligned(s, eb) || !aligned(codes, 4))
    return LMBP_EINVAL;
  const uint64_t b = uint64_t(n) * eb;
  const Span sg = span(g, b), su = span(u, b), sh = span(h, b), ss = span(s, b);
  const Span sc = span(codes, lmbp_codes_bytes(n));
  // h may replace g or u in place; s and codes overlap nothing.
  if (bad_pair(sg, su, false) || bad_pair(sh, sg, true) || bad_pair(sh, su, true) ||
      bad_pair(ss, sg, false) || bad_pair(ss, su, false) || bad_pair(ss, sh, false) ||
      bad_pair(sc, sg, false) || bad_pair(sc, su, false) || bad_pair(sc, sh, false) ||
      bad_pair(sc, ss, false))
    return LMBP_EOVERLAP;
  const bool vec_ok = aligned(g, 16) && aligned(u, 16) && aligned(h, 16) && aligned(s, 16);
  return from_hip(lmbp::launch_glu_fwd(lmbp::kSilu, dt == LMBP_BF16, n, g, u, h, s, codes, vec_ok,
                                       static_cast<hipStream_t>(stream)));
}

lmbp_status glu_bwd(lmbp_dtype dt, int64_t n, const void* dh, const void* u, const void* s,
                    const uint32_t* codes, void* dg, void* du, void* stream) {
  if (!known_dtype(dt)) return LMBP_EDTYPE;
  if (n < 0 || uint64_t(n) > (uint64_t(1) << 60)) return LMBP_EINVAL;
  if (n == 0) return LMBP_OK;
  if (!dh || !u || !s || !codes || !dg || !du) return LMBP_EINVAL;
  const int eb = elem_bytes(dt);
  if (!aligned(dh, eb) || !aligned(u, eb) || !aligned(s, eb) || !aligned(dg, eb) ||
      !aligned(du, eb) || !aligned(codes, 4))
    return LMBP_EINVAL;
  const uint64_t b = uint64_t(n) * eb;
  const Span sh = span(dh, b), su = span(u, b), ss = span(s, b), sg = span(dg, b), sd = span(du, b);
  const Span sc = span(codes, lmbp_codes_bytes(n));
  // dg may replace dh and du may replace u in place; nothing else overlaps.
  if (bad_pair(sh, su, false) || bad_pair(sh, ss, false) || bad_pair(su, ss, false) ||
      bad_pair(sg, sh, true) || bad_pair(sg, su, false) || bad_pair(sg, ss, false) ||
      bad_pair(sd, su, true) || bad_pair(sd, sh, false) || bad_pair(sd, ss, false) ||
      bad_pair(sd, sg, false) || bad_pair(sc, sh, false) || bad_pair(sc, su, false) ||
      bad_pair(sc, ss, false) || bad_pair(sc, sg, false) || bad_pair(sc, sd, false))
    return LMBP_EOVERLAP;
  const bool vec_ok = aligned(dh, 16) && aligned(u, 16) && aligned(s, 16) && aligned(dg, 16) &&
                      aligned(du, 16);
  return from_hip(lmbp::launch_glu_bwd(lmbp::kSilu, dt == LMBP_BF16, n, dh, u, s, codes, dg, du,
                                       vec_ok, static_cast<hipStream_t>(stream)));
}

uint64_t step_codes_bytes(int bits, int64_t n) {
  const uint64_t per = uint64_t(32 / bits);
  return n <= 0 ? 0 : (uint64_t(n) + per - 1) / per * 4;
}

bool valid_bits(int bits) { return bits >= 1 && bits <= 4; }

// Largest fp32 value not above c (for finite c within the fp32 range).
float round_down_f32(double c) {
  float f = static_cast<float>(c);
  if (static_cast<double>(f) > c) f = std::nextafter(f, -std::numeric_limits<float>::infinity());
  return f;
}

lmbp_status stepact_fwd_impl(int act, int bits, const double* thresholds, lmbp_dtype dt, int64_t n,
                             const void* x, void* y, uint32_t* codes, void* stream) {
  if (!known_dtype(dt)) return LMBP_EDTYPE;
  if (!valid_bits(bits) || (act != LMBP_ACT_GELU && act != LMBP_ACT_SILU)) return LMBP_EINVAL;
  if (n < 0 || uint64_t(n) > (uint64_t(1) << 60)) return LMBP_EINVAL;
  if (!thresholds) return LMBP_EINVAL;
  const int nt = (1 << bits) - 1;
  lmbp::StepTable tab{};
  for (int i = 0; i < nt; ++i) {
    const double c = thresholds[i];
    if (!std::isfinite(c) || std::fabs(c) > 3.0e38 || (i > 0 && !(c > thresholds[i - 1])))
      return LMBP_EINVAL;
    tab.t[i] = round_down_f32(c);
  }
  if (n == 0) return LMBP_OK;
  if (!x || !y || !codes) return LMBP_EINVAL;
  const int eb = elem_bytes(dt);
  if (!aligned(x, eb) || !aligned(y, eb) || !aligned(codes, 4)) return LMBP_EINVAL;
  const Span sx = span(x, uint64_t(n) * eb), sy = span(y, uint64_t(n) * eb);
  const Span sc = span(codes, step_codes_bytes(bits, n));
  if (bad_pair(sx, sy, true) || bad_pair(sc, sx, false) || bad_pair(sc, sy, false))
    return LMBP_EOVERLAP;
  const bool vec_ok = aligned(x, 16) && aligned(y, 16);
  return from_hip(lmbp::launch_stepact_fwd(act == LMBP_ACT_GELU ? lmbp::kGelu : lmbp::kSilu, bits,
                                           dt == LMBP_BF16, n, x, y, codes, vec_ok, tab,
                                           static_cast<hipStream_t>(stream)));
}

lmbp_status stepact_bwd_impl(int bits, const double* levels, lmbp_dtype dt, int64_t n, const void* dy,
                             const uint32_t* codes, void* dx, void* stream) {
  if (!known_dtype(dt)) return LMBP_EDTYPE;
  if (!valid_bits(bits)) return LMBP_EINVAL;
  if (n < 0 || uint64_t(n) > (uint64_t(1) << 60)) return LMBP_EINVAL;
  if (!levels) return LMBP_EINVAL;
  lmbp::StepTable tab{};
  for (int i = 0; i < (1 << bits); ++i) {
    if (!std::isfinite(levels[i]) || std::fabs(levels[i]) > 3.0e38) return LMBP_EINVAL;
    tab.lv[i] = static_cast<float>(levels[i]);
  }
  if (n == 0) return LMBP_OK;
  if (!dy || !dx || !codes) return LMBP_EINVAL;
  const int eb = elem_bytes(dt);
  if (!aligned(dy, eb) || !aligned(dx, eb) || !aligned(codes, 4)) return LMBP_EINVAL;
  const Span sg = span(dy, uint64_t(n) * eb), sd = span(dx, uint64_t(n) * eb);
  const Span sc = span(codes, step_codes_bytes(bits, n));
  if (bad_pair(sg, sd, true) || bad_pair(sc, sg, false) || bad_pair(sc, sd, false))
    return LMBP_EOVERLAP;
  const bool vec_ok = aligned(dy, 16) && aligned(dx, 16);
  return from_hip(lmbp::launch_stepact_bwd(bits, dt == LMBP_BF16, n, dy, codes, dx, vec_ok, tab,
                                           static_cast<hipStream_t>(stream)));
}

lmbp_status norm_fwd(bool ln, lmbp_dtype dt, int64_t rows, int64_t cols, float eps, const void* x,
                     void* z, float* rstd, void* stream) {
  if (!known_dtype(dt)) return LMBP_EDTYPE;
  if (rows < 0 || cols < 0) return LMBP_EINVAL;
  if (rows == 0) return LMBP_OK;
  if (cols == 0) return LMBP_EINVAL;
  if (!(std::isfinite(eps) && eps > 0.0f)) return LMBP_EINVAL;
  if (!x || !z || !rstd) return LMBP_EINVAL;
  const int eb = elem_bytes(dt);
  if (!aligned(x, eb) || !aligned(z, eb) || !aligned(rstd, 4)) return LMBP_EINVAL;
  if (uint64_t(rows) > (uint64_t(1) << 62) / uint64_t(cols) / 4) return LMBP_EINVAL;
  const uint64_t bytes = uint64_t(rows) * uint64_t(cols) * eb;
  const Span sx = span(x, bytes), sz = span(z, bytes), sr = span(rstd, uint64_t(rows) * 4);
  if (bad_pair(sx, sz, true) || bad_pair(sr, sx, false) || bad_pair(sr, sz, false))
    return LMBP_EOVERLAP;
  const bool vec_ok = aligned(x, 16) && aligned(z, 16) && (uint64_t(cols) * eb) % 16 == 0;
  return from_hip(lmbp::launch_norm_fwd(ln, dt == LMBP_BF16, rows, cols, eps, x, z, rstd, vec_ok,
                                        static_cast<hipStream_t>(stream)));
}

lmbp_status norm_bwd(bool ln, lmbp_dtype dt, int64_t rows, int64_t cols, const void* dz,
                     const void* z, const float* rstd, void* dx, void* stream) {
  if (!known_dtype(dt)) return LMBP_EDTYPE;
  if (rows < 0 || cols < 0) return LMBP_EINVAL;
  if (rows == 0) return LMBP_OK;
  if (cols == 0) return LMBP_EINVAL;
  if (!dz || !z || !rstd || !dx) return LMBP_EINVAL;
  const int eb = elem_bytes(dt);
  if (!aligned(dz, eb) || !aligned(z, eb) || !aligned(dx, eb) || !aligned(rstd, 4))
    return LMBP_EINVAL;
  if (uint64_t(rows) > (uint64_t(1) << 62) / uint64_t(cols) / 4) return LMBP_EINVAL;
  const uint64_t bytes = uint64_t(rows) * uint64_t(cols) * eb;
  const Span sg = span(dz, bytes), sz = span(z, bytes), sd = span(dx, bytes);
  const Span sr = span(rstd, uint64_t(rows) * 4);
  if (bad_pair(sg, sd, true) || bad_pair(sz, sd, false) || bad_pair(sr, sd, false) ||
      bad_pair(sr, sg, false) || bad_pair(sr, sz, false))
    return LMBP_EOVERLAP;
  const bool vec_ok = aligned(dz, 16) && aligned(z, 16) && aligned(dx, 16) &&
                      (uint64_t(cols) * eb) % 16 == 0;
  return from_hip(lmbp::launch_norm_bwd(ln, dt == LMBP_BF16, rows, cols, dz, z, rstd, dx, vec_ok,
                                        static_cast<hipStream_t>(stream)));
}

lmbp_status linear_act_fwd_impl(lmbp_act act, lmbp_dtype dt, int64_t m, int64_t n, int64_t k,
                                const void* x, const void* w, const void* bias, void* y,
                                uint32_t* codes, void* z, void* stream) {
  if (!known_dtype(dt)) return LMBP_EDTYPE;
  if (dt != LMBP_BF16) return LMBP_EDTYPE;
  if (act != LMBP_ACT_GELU && act != LMBP_ACT_SILU) return LMBP_EINVAL;
  const int64_t lim = int64_t(1) << 31;
  if (m < 0 || n < 0 || k < 0 || m >= lim || n >= lim || k >= lim) return LMBP_EINVAL;
  if (n % 16 != 0 || k % 8 != 0 || k > (int64_t(1) << 21)) return LMBP_EINVAL;
  if (m == 0 || n == 0) return LMBP_OK;
  if (uint64_t(m) * uint64_t(n) > (uint64_t(1) << 60)) return LMBP_EINVAL;
  if (!y || !codes || (k > 0 && (!x || !w))) return LMBP_EINVAL;
  if ((x && !aligned(x, 16)) || (w && !aligned(w, 16)) || !aligned(y, 16) || (z && !aligned(z, 16)) ||
      !aligned(codes, 4) || (bias && !aligned(bias, 2)))
    return LMBP_EINVAL;
  const uint64_t mn = uint64_t(m) * uint64_t(n);
  const Span sy = span(y, mn * 2), sc = span(codes, lmbp_codes_bytes(int64_t(mn)));
  const Span sz = span(z, z ? mn * 2 : 0);
  const Span ins[3] = {span(x, x ? uint64_t(m) * uint64_t(k) * 2 : 0),
                       span(w, w ? uint64_t(n) * uint64_t(k) * 2 : 0),
                       span(bias, bias ? uint64_t(n) * 2 : 0)};
  const Span outs[3] = {sy, sc, sz};
  for (int i = 0; i < 3; ++i) {
    for (int j = i + 1; j < 3; ++j)
      if (overlaps(outs[i], outs[j])) return LMBP_EOVERLAP;
    for (const Span& in : ins)
      if (overlaps(outs[i], in)) return LMBP_EOVERLAP;
  }
  return from_hip(lmbp::launch_linear_act_fwd(act == LMBP_ACT_GELU ? lmbp::kGelu : lmbp::kSilu, m,
                                              n, k, x, w, bias, y, codes, z,
                                              static_cast<hipStream_t>(stream)));
}

lmbp_status linear_swiglu_fwd_impl(lmbp_dtype dt, int64_t m, int64_t n, int64_t k, const void* x,
                                   const void* w_gate, const void* w_up, void* h, void* s, void* u,
                                   uint32_t* codes, void* g, void* stream) {
  if (!known_dtype(dt) || dt != LMBP_BF16) return LMBP_EDTYPE;
  const int64_t lim = int64_t(1) << 31;
  if (m < 0 || n < 0 || k < 0 || m >= lim || n >= lim || k >= lim) return LMBP_EINVAL;
  if (n % 16 != 0 || k % 8 != 0 || k > (int64_t(1) << 21)) return LMBP_EINVAL;
  if (m == 0 || n == 0) return LMBP_OK;
  if (uint64_t(m) * uint64_t(n) > (uint64_t(1) << 60)) return LMBP_EINVAL;
  if (!h || !s || !u || !codes || (k > 0 && (!x || !w_gate || !w_up))) return LMBP_EINVAL;
  const void* sixteen[] = {x, w_gate, w_up, h, s, u, g};
  for (const void* p : sixteen)
    if (p && !aligned(p, 16)) return LMBP_EINVAL;
  if (!aligned(codes, 4)) return LMBP_EINVAL;
  const uint64_t mn = uint64_t(m) * uint64_t(n);
  const Span outs[5] = {span(h, mn * 2), span(s, mn * 2), span(u, mn * 2),
                        span(codes, lmbp_codes_bytes(int64_t(mn))), span(g, g ? mn * 2 : 0)};
  const Span ins[3] = {span(x, x ? uint64_t(m) * uint64_t(k) * 2 : 0),
                       span(w_gate, w_gate ? uint64_t(n) * uint64_t(k) * 2 : 0),
                       span(w_up, w_up ? uint64_t(n) * uint64_t(k) * 2 : 0)};
  for (int i = 0; i < 5; ++i) {
    for (int j = i + 1; j < 5; ++j)
      if (overlaps(outs[i], outs[j])) return LMBP_EOVERLAP;
    for (const Span& in : ins)
      if (overlaps(outs[i], in)) return LMBP_EOVERLAP;
  }
  return from_hip(lmbp::launch_linear_glu_fwd(m, n, k, x, w_gate, w_up, h, s, u, codes, g,
                                              static_cast<hipStream_t>(stream)));
}

// The norm-in-front forms: x [m x k] is MS-RMSNorm's input, z [m x k] and rstd [m] its
// outputs; the rest as for the plain forms. k >= 8 (a norm needs a row).
lmbp_status check_norm_in_front(int64_t m, int64_t n, int64_t k, float eps, const void* x,
                                const void* z, const float* rstd) {
  const int64_t lim = int64_t(1) << 31;
  if (m < 0 || n < 0 || k < 0 || m >= lim || n >= lim || k >= lim) return LMBP_EINVAL;
  if (n % 16 != 0 || k % 8 != 0 || k > (int64_t(1) << 21)) return LMBP_EINVAL;
  if (!(std::isfinite(eps) && eps > 0.0f)) return LMBP_EINVAL;
  if (m > 0 && k == 0) return LMBP_EINVAL;
  if (m > 0 && (!x || !z || !rstd)) return LMBP_EINVAL;
  if ((x && !aligned(x, 16)) || (z && !aligned(z, 16)) || (rstd && !aligned(rstd, 4))) return LMBP_EINVAL;
  if (m == 0) return LMBP_OK;
  const uint64_t mk = uint64_t(m) * uint64_t(k);
  const Span sx = span(x, mk * 2), sz = span(z, mk * 2), sr = span(rstd, uint64_t(m) * 4);
  if (overlaps(sx, sz) || overlaps(sx, sr) || overlaps(sz, sr)) return LMBP_EOVERLAP;
  return LMBP_OK;
}

// A layer with no output features (n == 0) still normalises its input: z and rstd come
// from the stand-alone norm kernel (the same bytes the fused path writes).
hipError_t norm_in_front_only(int64_t m, int64_t k, float eps, const void* x, void* z, float* rstd,
                              void* stream) {
  return lmbp::launch_norm_fwd(false, true, m, k, eps, x, z, rstd, true,
                               static_cast<hipStream_t>(stream));
}

lmbp_status msrms_linear_act_fwd_impl(lmbp_act act, lmbp_dtype dt, int64_t m, int64_t n, int64_t k,
                                      float eps, const void* x, const void* w, const void* bias,
                                      void* y, uint32_t* codes, void* pre, void* z, float* rstd,
                                      void* stream) {
  if (!known_dtype(dt) || dt != LMBP_BF16) return LMBP_EDTYPE;
  if (act != LMBP_ACT_GELU && act != LMBP_ACT_SILU) return LMBP_EINVAL;
  const lmbp_status st = check_norm_in_front(m, n, k, eps, x, z, rstd);
  if (st != LMBP_OK) return st;
  if (m == 0) return LMBP_OK;
  if (n == 0) return from_hip(norm_in_front_only(m, k, eps, x, z, rstd, stream));
  if (uint64_t(m) * uint64_t(n) > (uint64_t(1) << 60)) return LMBP_EINVAL;
  if (!y || !codes || !w) return LMBP_EINVAL;
  if (!aligned(w, 16) || !aligned(y, 16) || !aligned(codes, 4) || (bias && !aligned(bias, 2)) ||
      (pre && !aligned(pre, 16)))
    return LMBP_EINVAL;
  const uint64_t mn = uint64_t(m) * uint64_t(n), mk = uint64_t(m) * uint64_t(k);
  const Span outs[5] = {span(y, mn * 2), span(codes, lmbp_codes_bytes(int64_t(mn))), span(z, mk * 2),
                        span(rstd, uint64_t(m) * 4), span(pre, pre ? mn * 2 : 0)};
  const Span ins[3] = {span(x, mk * 2), span(w, uint64_t(n) * uint64_t(k) * 2),
                       span(bias, bias ? uint64_t(n) * 2 : 0)};
  for (int i = 0; i < 5; ++i) {
    for (int j = i + 1; j < 5; ++j)
      if (overlaps(outs[i], outs[j])) return LMBP_EOVERLAP;
    for (const Span& in : ins)
      if (overlaps(outs[i], in)) return LMBP_EOVERLAP;
  }
  return from_hip(lmbp::launch_linear_rms_act_fwd(act == LMBP_ACT_GELU ? lmbp::kGelu : lmbp::kSilu, m, n,
                                                  k, eps, x, w, bias, y, codes, pre, z, rstd,
                                                  static_cast<hipStream_t>(stream)));
}

lmbp_status msrms_linear_swiglu_fwd_impl(lmbp_dtype dt, int64_t m, int64_t n, int64_t k, float eps,
                                         const void* x, const void* w_gate, const void* w_up, void* h,
                                         void* s, void* u, uint32_t* codes, void* g, void* z,
                                         float* rstd, void* stream) {
  if (!known_dtype(dt) || dt != LMBP_BF16) return LMBP_EDTYPE;
  const lmbp_status st = check_norm_in_front(m, n, k, eps, x, z, rstd);
  if (st != LMBP_OK) return st;
  if (m == 0) return LMBP_OK;
  if (n == 0) return from_hip(norm_in_front_only(m, k, eps, x, z, rstd, stream));
  if (uint64_t(m) * uint64_t(n) > (uint64_t(1) << 60)) return LMBP_EINVAL;
  if (!h || !s || !u || !codes || !w_gate || !w_up) return LMBP_EINVAL;
  const void* sixteen[] = {w_gate, w_up, h, s, u};
  for (const void* p : sixteen)
    if (!aligned(p, 16)) return LMBP_EINVAL;
  if (!aligned(codes, 4) || (g && !aligned(g, 16))) return LMBP_EINVAL;
  const uint64_t mn = uint64_t(m) * uint64_t(n), mk = uint64_t(m) * uint64_t(k);
  const Span outs[7] = {span(h, mn * 2), span(s, mn * 2), span(u, mn * 2),
                        span(codes, lmbp_codes_bytes(int64_t(mn))), span(z, mk * 2),
                        span(rstd, uint64_t(m) * 4), span(g, g ? mn * 2 : 0)};
  const Span ins[3] = {span(x, mk * 2), span(w_gate, uint64_t(n) * uint64_t(k) * 2),
                       span(w_up, uint64_t(n) * uint64_t(k) * 2)};
  for (int i = 0; i < 7; ++i) {
    for (int j = i + 1; j < 7; ++j)
      if (overlaps(outs[i], outs[j])) return LMBP_EOVERLAP;
    for (const Span& in : ins)
      if (overlaps(outs[i], in)) return LMBP_EOVERLAP;
  }
  return from_hip(lmbp::launch_linear_rms_glu_fwd(m, n, k, eps, x, w_gate, w_up, h, s, u, codes, g, z,
                                                  rstd, static_cast<hipStream_t>(stream)));
}

}  // namespace

extern "C" {

size_t lmbp_codes_bytes(int64_t n) { return n <= 0 ? 0 : size_t((uint64_t(n) + 15) / 16) * 4; }

const char* lmbp_strerror(lmbp_status st) {
  switch (st) {
    case LMBP_OK: return "success";
    case LMBP_EINVAL: return "invalid argument (size, pointer, alignment or eps)";
    case LMBP_EDTYPE: return "unknown dtype";
    case LMBP_EOVERLAP: return "buffers overlap in a way the call does not allow";
    case LMBP_EHIP: return "HIP kernel launch failed";
  }
  return "unknown status";
}

int lmbp_last_hip_error(void) { return g_last_hip_error; }

lmbp_status regelu2_fwd(lmbp_dtype dt, int64_t n, const void* x, void* y, uint32_t* codes,
                        void* stream) {
  return act_fwd(lmbp::kGelu, dt, n, x, y, codes, stream);
}
lmbp_status regelu2_bwd(lmbp_dtype dt, int64_t n, const void* dy, const uint32_t* codes, void* dx,
                        void* stream) {
  return act_bwd(lmbp::kGelu, dt, n, dy, codes, dx, stream);
}
lmbp_status resilu2_fwd(lmbp_dtype dt, int64_t n, const void* x, void* y, uint32_t* codes,
                        void* stream) {
  return act_fwd(lmbp::kSilu, dt, n, x, y, codes, stream);
}
lmbp_status resilu2_bwd(lmbp_dtype dt, int64_t n, const void* dy, const uint32_t* codes, void* dx,
                        void* stream) {
  return act_bwd(lmbp::kSilu, dt, n, dy, codes, dx, stream);
}

lmbp_status reswiglu2_fwd(lmbp_dtype dt, int64_t n, const void* g, const void* u, void* h, void* s,
                          uint32_t* codes, void* stream) {
  return glu_fwd(dt, n, g, u, h, s, codes, stream);
}
lmbp_status reswiglu2_bwd(lmbp_dtype dt, int64_t n, const void* dh, const void* u, const void* s,
                          const uint32_t* codes, void* dg, void* du, void* stream) {
  return glu_bwd(dt, n, dh, u, s, codes, dg, du, stream);
}

size_t lmbp_stepact_codes_bytes(int bits, int64_t n) {
  return valid_bits(bits) ? size_t(step_codes_bytes(bits, n)) : 0;
}
lmbp_status stepact_fwd(lmbp_act act, int bits, const double* thresholds, lmbp_dtype dt, int64_t n,
                        const void* x, void* y, uint32_t* codes, void* stream) {
  return stepact_fwd_impl(act, bits, thresholds, dt, n, x, y, codes, stream);
}
lmbp_status stepact_bwd(int bits, const double* levels, lmbp_dtype dt, int64_t n, const void* dy,
                        const uint32_t* codes, void* dx, void* stream) {
  return stepact_bwd_impl(bits, levels, dt, n, dy, codes, dx, stream);
}

lmbp_status msln_fwd(lmbp_dtype dt, int64_t rows, int64_t cols, float eps, const void* x, void* z,
                     float* rstd, void* stream) {
  return norm_fwd(true, dt, rows, cols, eps, x, z, rstd, stream);
}
lmbp_status msln_bwd(lmbp_dtype dt, int64_t rows, int64_t cols, const void* dz, const void* z,
                     const float* rstd, void* dx, void* stream) {
  return norm_bwd(true, dt, rows, cols, dz, z, rstd, dx, stream);
}
lmbp_status msrms_fwd(lmbp_dtype dt, int64_t rows, int64_t cols, float eps, const void* x, void* z,
                      float* rstd, void* stream) {
  return norm_fwd(false, dt, rows, cols, eps, x, z, rstd, stream);
}
lmbp_status msrms_bwd(lmbp_dtype dt, int64_t rows, int64_t cols, const void* dz, const void* z,
                      const float* rstd, void* dx, void* stream) {
  return norm_bwd(false, dt, rows, cols, dz, z, rstd, dx, stream);
}

lmbp_status linear_act_fwd(lmbp_act act, lmbp_dtype dt, int64_t m, int64_t n, int64_t k,
                           const void* x, const void* w, const void* bias, void* y,
                           uint32_t* codes, void* z, void* stream) {
  return linear_act_fwd_impl(act, dt, m, n, k, x, w, bias, y, codes, z, stream);
}

lmbp_status linear_swiglu_fwd(lmbp_dtype dt, int64_t m, int64_t n, int64_t k, const void* x,
                              const void* w_gate, const void* w_up, void* h, void* s, void* u,
                              uint32_t* codes, void* g, void* stream) {
  return linear_swiglu_fwd_impl(dt, m, n, k, x, w_gate, w_up, h, s, u, codes, g, stream);
}

lmbp_status msrms_linear_act_fwd(lmbp_act act, lmbp_dtype dt, int64_t m, int64_t n, int64_t k, float eps,
                                 const void* x, const void* w, const void* bias, void* y, uint32_t* codes,
                                 void* pre, void* z, float* rstd, void* stream) {
  return msrms_linear_act_fwd_impl(act, dt, m, n, k, eps, x, w, bias, y, codes, pre, z, rstd, stream);
}

lmbp_status msrms_linear_swiglu_fwd(lmbp_dtype dt, int64_t m, int64_t n, int64_t k, float eps,
                                    const void* x, const void* w_gate, const void* w_up, void* h, void* s,
                                    void* u, uint32_t* codes, void* g, void* z, float* rstd, void* stream) {
  return msrms_linear_swiglu_fwd_impl(dt, m, n, k, eps, x, w_gate, w_up, h, s, u, codes, g, z, rstd,
                                      stream);
}

lmbp_status lmbp_copy(const void* src, void* dst, int64_t bytes, void* stream) {
  if (bytes < 0) return LMBP_EINVAL;
  if (bytes == 0) return LMBP_OK;
  if (!src || !dst || !aligned(src, 16) || !aligned(dst, 16)) return LMBP_EINVAL;
  if (overlaps(span(src, uint64_t(bytes)), span(dst, uint64_t(bytes)))) return LMBP_EOVERLAP;
  return from_hip(lmbp::launch_copy(src, dst, bytes, static_cast<hipStream_t>(stream)));
}

}  // extern "C"
