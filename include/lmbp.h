/*
 * lmbp.h - C ABI of the low-memory backpropagation kernels for AMD MI355X (gfx950).
 *
 * Operations from "Reducing Fine-Tuning Memory Overhead by Approximate and
 * Memory-Sharing Backpropagation" (Yang et al., ICML 2024):
 *
 *   regelu2_fwd / regelu2_bwd   ReGELU2  (Sec. 4.2; constants Appendix E)
 *   resilu2_fwd / resilu2_bwd   ReSiLU2  (Sec. 4.2; constants Appendix E)
 *   msln_fwd    / msln_bwd      MS-LN    (Sec. 5.2 Alg. 1; Appendix G Alg. 2)
 *   msrms_fwd   / msrms_bwd     MS-RMSNorm (Appendix G Alg. 3)
 *   reswiglu2_fwd / reswiglu2_bwd  ReSiLU2 fused with the SwiGLU product (LLaMA MLP)
 *   stepact_fwd / stepact_bwd      k-bit family members with runtime tables (ReGELU2-d, ...)
 *   linear_act_fwd                 a linear layer whose output goes through ReGELU2 /
 *                                  ReSiLU2, fused (the pre-activation stays on chip)
 *   linear_swiglu_fwd              the LLaMA MLP's two projections + SwiGLU, fused
 *   msrms_linear_act_fwd           MS-RMSNorm, the merged linear layer and ReGELU2 /
 *                                  ReSiLU2 forward, fused (the norm in the GEMM)
 *   msrms_linear_swiglu_fwd        MS-RMSNorm and the LLaMA MLP's input side, fused
 *
 * Conventions shared by every call
 * --------------------------------
 * - Pointers are device pointers (HBM) owned and allocated by the caller; the
 *   library never allocates, frees or synchronizes. Every call only enqueues
 *   kernels on `stream` (a hipStream_t; NULL means the null stream) and returns.
 * - Tensors are dense and row-major. Activation ops see a flat tensor of n
 *   elements; norm ops see `rows` rows of `cols` elements (cols = the normalized
 *   width p of the paper).
 * - dtype selects the storage of every floating-point tensor argument except the
 *   norm statistic `rstd`, which is always fp32. Arithmetic is fp32 in all cases.
 * - Pointers need only element alignment (2 bytes for bf16, 4 for fp32 and for
 *   codes / rstd); 16-byte aligned tensors whose rows are multiples of 16 bytes
 *   take the vectorized path, anything else a slower general path with the same
 *   results up to floating-point summation order.
 * - Aliasing: only the exact in-place pairs named for each call are allowed
 *   (same start address, same size). Any other overlap of two buffers of a call
 *   returns LMBP_EOVERLAP before anything is launched.
 * - Errors are checked on the host before any launch: LMBP_EINVAL for negative
 *   sizes, cols == 0 with rows > 0, a NULL pointer with a nonzero size, a
 *   misaligned pointer, or eps not finite and > 0; LMBP_EDTYPE for an unknown
 *   dtype. n == 0 or rows == 0 is a successful no-op. LMBP_EHIP means the kernel
 *   launch failed; lmbp_last_hip_error() then returns the hipError_t value for the
 *   calling thread. No C++ exception crosses this interface.
 * - Results are deterministic: no atomics, fixed reduction order.
 */
#ifndef LMBP_H
#define LMBP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { LMBP_FP32 = 0, LMBP_BF16 = 1 } lmbp_dtype;

typedef enum {
  LMBP_OK = 0,
  LMBP_EINVAL = 1,
  LMBP_EDTYPE = 2,
  LMBP_EOVERLAP = 3,
  LMBP_EHIP = 4
} lmbp_status;

/* Bytes of the packed code buffer for n activation elements: 4 * ceil(n / 16).
 * The code of flat element i occupies bits [2(i mod 16), 2(i mod 16) + 1] of 32-bit
 * word i / 16 (least significant bits first); unused bits of the last word are 0.
 * Returns 0 for n <= 0. */
size_t lmbp_codes_bytes(int64_t n);

/* Static description of a status code. */
const char *lmbp_strerror(lmbp_status st);

/* hipError_t recorded by the last call on this thread that returned LMBP_EHIP. */
int lmbp_last_hip_error(void);

/* ------------------------------------------------------------------------
 * ReGELU2 / ReSiLU2 (Sec. 4.2, eq. relus_family with k = 2).
 *
 * Forward: y = GELU(x) = x/2 (1 + erf(x / sqrt 2))   (regelu2)
 *          y = SiLU(x) = x / (1 + e^-x)              (resilu2)
 * computed exactly (fp32 arithmetic), plus the 2-bit code of every element: the
 * number of the three biases c1 < c2 < c3 of Appendix E lying strictly below x.
 * Backward: dx = dy * s[code], where s = (0, a1, a1 + a2, 1) is the slope of the
 * three-ReLU combination on each of its four segments (Prop. 4.3).
 *
 *   x, y   : n elements of dtype. y == x (in place) is allowed.
 *   codes  : lmbp_codes_bytes(n) bytes, 4-byte aligned, written completely
 *            (including zero tail bits); must not overlap x or y.
 *   dy, dx : n elements of dtype. dx == dy is allowed.
 *   codes (bwd): as written by the matching forward; read only.
 * ------------------------------------------------------------------------ */
lmbp_status regelu2_fwd(lmbp_dtype dt, int64_t n, const void *x, void *y,
                        uint32_t *codes, void *stream);
lmbp_status regelu2_bwd(lmbp_dtype dt, int64_t n, const void *dy,
                        const uint32_t *codes, void *dx, void *stream);
lmbp_status resilu2_fwd(lmbp_dtype dt, int64_t n, const void *x, void *y,
                        uint32_t *codes, void *stream);
lmbp_status resilu2_bwd(lmbp_dtype dt, int64_t n, const void *dy,
                        const uint32_t *codes, void *dx, void *stream);

/* ------------------------------------------------------------------------
 * ReSiLU2 inside a SwiGLU product, h = SiLU(g) * u: the LLaMA MLP, where the paper
 * substitutes ReSiLU2 for SiLU (Sec. 6). The backward is the Approx-BP backward of
 * the product (Sec. 4.1): the exact product rule on the saved forward activation
 * s = SiLU(g), and the step derivative of the three-ReLU combination for SiLU.
 *
 * Forward:  s = SiLU(g), h = s * u, codes of g (as resilu2_fwd).
 * Backward: dg = dh * u * s[code],  du = dh * s.
 *
 *   g, u   : n elements of dtype (inputs). h: n elements (output; h == g or h == u
 *            allowed). s: n elements (output, saved for the backward; overlaps
 *            nothing). codes: lmbp_codes_bytes(n) bytes (output; overlaps nothing).
 *   dh, u, s, codes (bwd): inputs; dg, du: n elements (outputs; dg == dh and
 *            du == u allowed, no other overlap).
 * Saved state per element: the 2-bit code plus s (which the product keeps anyway);
 * g itself is not needed.
 * ------------------------------------------------------------------------ */
lmbp_status reswiglu2_fwd(lmbp_dtype dt, int64_t n, const void *g, const void *u,
                          void *h, void *s, uint32_t *codes, void *stream);
lmbp_status reswiglu2_bwd(lmbp_dtype dt, int64_t n, const void *dh, const void *u,
                          const void *s, const uint32_t *codes, void *dg, void *du,
                          void *stream);

/* ------------------------------------------------------------------------
 * General members of the ReLU-combination family (eq. relus_family with k bits;
 * Appendix I's ReGELU2-d is k = 2 with other constants), with runtime tables.
 *
 * Forward: y = GELU(x) or SiLU(x) exactly (act), and the k-bit code of every
 * element: the number of the 2^k - 1 thresholds strictly below x (the biases c of
 * the combination). Backward: dx = dy * levels[code] (2^k levels: the slopes of the
 * combination on its segments, cumulative sums of its weights).
 *
 *   bits       : k in {1, 2, 3, 4}; codes hold floor(32/k) elements per 32-bit word
 *                (32, 16, 10, 8), least significant first (code j of a word at bits
 *                k j .. k j + k - 1; for k = 3 the top two bits are 0), zero tail;
 *                lmbp_stepact_codes_bytes(k, n) bytes.
 *   thresholds : host array of 2^k - 1 finite, strictly increasing doubles (read
 *                during the call only). Each is applied as an exact real comparison.
 *   levels     : host array of 2^k finite doubles, used as fp32 values.
 *   x, y, dy, dx, codes: as for regelu2_fwd / regelu2_bwd (y == x, dx == dy allowed).
 * LMBP_EINVAL also for bad k, act, tables or a NULL table pointer.
 * ------------------------------------------------------------------------ */
typedef enum { LMBP_ACT_GELU = 0, LMBP_ACT_SILU = 1 } lmbp_act;

size_t lmbp_stepact_codes_bytes(int bits, int64_t n);
lmbp_status stepact_fwd(lmbp_act act, int bits, const double *thresholds, lmbp_dtype dt,
                        int64_t n, const void *x, void *y, uint32_t *codes, void *stream);
lmbp_status stepact_bwd(int bits, const double *levels, lmbp_dtype dt, int64_t n,
                        const void *dy, const uint32_t *codes, void *dx, void *stream);

/* ------------------------------------------------------------------------
 * MS-LN (Sec. 5.2 Alg. 1, Appendix G Alg. 2) and MS-RMSNorm (Alg. 3), for a
 * norm whose affine (alpha, beta) has been merged into the following linear
 * layer (W~ = W diag(alpha), b~ = W beta + b). Per row x of width p = cols:
 *
 * Forward:  sigma = sqrt(p^-1 |H x|^2 + eps),  z = H x / sigma,  rstd = 1 / sigma,
 *           with H x = x - mean(x) for MS-LN and H x = x for MS-RMSNorm.
 * Backward: dx = rstd * (H dz - z * mean(z * dz))   (= sigma^-1 (H - p^-1 z z^T) dz),
 *           computed from the saved output z and rstd only.
 *
 *   x, z    : rows x cols of dtype. z == x (in place) is allowed. z is the
 *             tensor the next (merged) linear layer keeps anyway.
 *   rstd    : rows fp32 values; must not overlap x, z, dz or dx.
 *   eps     : finite, > 0 (the paper uses 1e-6 or 1e-8; LLaMA-style RMSNorm 1e-5).
 *   dz, dx  : rows x cols of dtype. dx == dz is allowed; dx must not overlap z.
 * ------------------------------------------------------------------------ */
lmbp_status msln_fwd(lmbp_dtype dt, int64_t rows, int64_t cols, float eps,
                     const void *x, void *z, float *rstd, void *stream);
lmbp_status msln_bwd(lmbp_dtype dt, int64_t rows, int64_t cols, const void *dz,
                     const void *z, const float *rstd, void *dx, void *stream);
lmbp_status msrms_fwd(lmbp_dtype dt, int64_t rows, int64_t cols, float eps,
                      const void *x, void *z, float *rstd, void *stream);
lmbp_status msrms_bwd(lmbp_dtype dt, int64_t rows, int64_t cols, const void *dz,
                      const void *z, const float *rstd, void *dx, void *stream);

/* ------------------------------------------------------------------------
 * Linear layer followed by ReGELU2 / ReSiLU2 (Sec. 4.2), forward, fused: the
 * activation runs in the epilogue of the matrix product, so the pre-activation z,
 * which the backward pass of ReGELU2 / ReSiLU2 does not need (it keeps only the
 * codes), never has to be written out.
 *
 *   z = bf16( x W^T + b )        products accumulated in fp32, bias added in fp32,
 *                                one rounding to bf16 (nearest even)
 *   y = act(z), codes = 2-bit codes of z, exactly as regelu2_fwd / resilu2_fwd
 *   compute them from a stored z (same bytes).
 *
 *   dt     : LMBP_BF16 only (LMBP_EDTYPE otherwise).
 *   act    : LMBP_ACT_GELU (ReGELU2) or LMBP_ACT_SILU (ReSiLU2).
 *   m,n,k  : x is m x k, w is n x k (the weight of a linear layer, row-major), y and
 *            z are m x n. n must be a multiple of 16 (each row of codes fills whole
 *            words) and k a multiple of 8 with k <= 2^21; m, n >= 0, k >= 0 (k == 0
 *            gives z = b).
 *   x, w, y, z : 16-byte aligned.
 *   bias   : n bf16 values, or NULL for none.
 *   codes  : lmbp_codes_bytes(m * n) bytes, codes of the flattened m x n output.
 *   z      : NULL (not stored) or m x n bf16.
 * y, codes and z must not overlap each other or any input. The backward pass is
 * regelu2_bwd / resilu2_bwd on the codes followed by the two products of a linear
 * layer's backward.
 * ------------------------------------------------------------------------ */
lmbp_status linear_act_fwd(lmbp_act act, lmbp_dtype dt, int64_t m, int64_t n, int64_t k,
                           const void *x, const void *w, const void *bias, void *y,
                           uint32_t *codes, void *z, void *stream);

/* ------------------------------------------------------------------------
 * The gated form of the same fusion, for the LLaMA MLP (Sec. 6; ReSiLU2 inside
 * SwiGLU as in reswiglu2_fwd): both projections of the MLP's input and the SwiGLU
 * product in one kernel, the gate pre-activation g never written out.
 *
 *   g = bf16( x Wg^T ),  u = bf16( x Wu^T )   (fp32 accumulation, one rounding each)
 *   h = SiLU(g) * u,  s = SiLU(g),  codes of g — exactly what reswiglu2_fwd computes
 *   from stored g and u (same bytes); u is written too, since the backward needs it.
 *
 *   dt : LMBP_BF16 only. m, n, k, alignment and limits as for linear_act_fwd.
 *   x [m x k]; w_gate, w_up [n x k]; h, s, u [m x n]; codes of the m x n output;
 *   g : NULL (not stored) or m x n.
 * Outputs must not overlap each other or any input. Backward: reswiglu2_bwd on
 * (dh, u, s, codes), then the two linear layers' products.
 * ------------------------------------------------------------------------ */
lmbp_status linear_swiglu_fwd(lmbp_dtype dt, int64_t m, int64_t n, int64_t k, const void *x,
                              const void *w_gate, const void *w_up, void *h, void *s, void *u,
                              uint32_t *codes, void *g, void *stream);

/* ------------------------------------------------------------------------
 * MS-RMSNorm in front of the fused linear layer (Sec. 5.2 eq. norm_linear, App. G
 * Alg. 3): the norm's affine merged into W (and b), the normalised row z consumed by
 * the linear layer and kept as the saved tensor of both.
 *
 *   rstd = 1 / sqrt(p^-1 |x|^2 + eps) per row of x (p = k), fp32;
 *   z    = bf16( x rstd )              the norm's output: the same bytes (and rstd the
 *                                      same bits) as msrms_fwd computes from x;
 *   y, codes as linear_act_fwd / linear_swiglu_fwd, with the pre-activation
 *        bf16( rstd (x W^T) + b )      i.e. the row scale is applied to the fp32 sums of
 *                                      the products of x, before the bias: the linear
 *                                      layer sees the normalised row before its storage
 *                                      rounding (equal to z W^T + b in exact arithmetic;
 *                                      not byte-equal to linear_act_fwd applied to z).
 *
 * One statistics pass over x writes rstd; then the GEMM runs on x, and after their K
 * loops its blocks also write z (each row tile's columns shared out among the blocks of
 * that row, x read again from the caches), so the norm's output traffic overlaps the
 * matrix products of other blocks.
 *
 *   dt   : LMBP_BF16 only.
 *   m,n,k, x, w, bias, y, codes : as linear_act_fwd, with k >= 8 when m > 0.
 *   eps  : finite and > 0 (as msrms_fwd).
 *   pre  : NULL (not stored) or m x n bf16: the rounded pre-activation, from which y
 *          and codes are exactly what regelu2_fwd / resilu2_fwd compute (as
 *          linear_act_fwd's z).
 *   z    : m x k bf16, 16-byte aligned (required: the saved tensor).
 *   rstd : m fp32, 4-byte aligned.
 * n == 0 (no output features) still writes z and rstd, by the stand-alone norm kernel;
 * w, bias, y, codes and pre are then not used. m == 0 is a successful no-op.
 * No output may overlap another output or an input. The backward pass is the linear
 * layer's (or SwiGLU's) backward on the kept tensors, then msrms_bwd(dz, z, rstd).
 * ------------------------------------------------------------------------ */
lmbp_status msrms_linear_act_fwd(lmbp_act act, lmbp_dtype dt, int64_t m, int64_t n, int64_t k,
                                 float eps, const void *x, const void *w, const void *bias,
                                 void *y, uint32_t *codes, void *pre, void *z, float *rstd,
                                 void *stream);

/* The gated form: MS-RMSNorm, then linear_swiglu_fwd's two projections and SwiGLU
 * (g and u each bf16(rstd (x W^T))), z and rstd as above; h, s, u, codes and the
 * optional g (NULL: not stored) as linear_swiglu_fwd. */
lmbp_status msrms_linear_swiglu_fwd(lmbp_dtype dt, int64_t m, int64_t n, int64_t k, float eps,
                                    const void *x, const void *w_gate, const void *w_up, void *h,
                                    void *s, void *u, uint32_t *codes, void *g, void *z,
                                    float *rstd, void *stream);

/* ------------------------------------------------------------------------
 * Measurement utility (not part of the method): copies `bytes` bytes from src
 * to dst with 16-byte non-temporal vector loads and non-temporal device-scope vector
 * stores (written through the L2), the fastest plain copy measured on the GPU for
 * tensors of 32 MiB and more. src and dst must be 16-byte
 * aligned and must not overlap. Used as the plain-copy reference for bandwidth
 * and hardware-counter calibration.
 * ------------------------------------------------------------------------ */
lmbp_status lmbp_copy(const void *src, void *dst, int64_t bytes, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* LMBP_H */
