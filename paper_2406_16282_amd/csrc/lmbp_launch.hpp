// Internal launcher declarations between the C ABI layer and the kernel files.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lmbp {

enum { kGelu = 0, kSilu = 1 };

// Runtime tables of a general family member (kernel argument, passed by value):
// thresholds t[0..2^k-2] as fp32 round-down values, levels lv[0..2^k-1] in fp32.
struct StepTable {
  float t[15];
  float lv[16];
};

hipError_t launch_act_fwd(int act, bool bf16, int64_t n, const void* x, void* y,
                          uint32_t* codes, bool vec_ok, hipStream_t s);
hipError_t launch_act_bwd(int act, bool bf16, int64_t n, const void* dy, const uint32_t* codes,
                          void* dx, bool vec_ok, hipStream_t s);

// Gated form h = act(g) * u (only act = kSilu is instantiated).
hipError_t launch_glu_fwd(int act, bool bf16, int64_t n, const void* g, const void* u, void* h,
                          void* s, uint32_t* codes, bool vec_ok, hipStream_t st);
hipError_t launch_glu_bwd(int act, bool bf16, int64_t n, const void* dh, const void* u,
                          const void* s, const uint32_t* codes, void* dg, void* du, bool vec_ok,
                          hipStream_t st);

// vec_ok: every tensor pointer 16-byte aligned and cols * element bytes a
// multiple of 16 (each row starts on a vector boundary). A null z computes rstd only.
hipError_t launch_norm_fwd(bool ln, bool bf16, int64_t rows, int64_t cols, float eps,
                           const void* x, void* z, float* rstd, bool vec_ok, hipStream_t s);
hipError_t launch_norm_bwd(bool ln, bool bf16, int64_t rows, int64_t cols, const void* dz,
                           const void* z, const float* rstd, void* dx, bool vec_ok,
                           hipStream_t s);

hipError_t launch_stepact_fwd(int act, int bits, bool bf16, int64_t n, const void* x, void* y,
                              uint32_t* codes, bool vec_ok, const StepTable& tab, hipStream_t s);
hipError_t launch_stepact_bwd(int bits, bool bf16, int64_t n, const void* dy, const uint32_t* codes,
                              void* dx, bool vec_ok, const StepTable& tab, hipStream_t s);

// z = bf16(x W^T + bias) (bf16 operands, fp32 accumulation); y = act(z), codes of z;
// z stored when non-null. N % 16 == 0, K % 8 == 0, x/w/y/z 16-byte aligned.
hipError_t launch_linear_act_fwd(int act, int64_t M, int64_t N, int64_t K, const void* x,
                                 const void* w, const void* bias, void* y, uint32_t* codes,
                                 void* z, hipStream_t s);

// Gated form: g = bf16(x Wg^T), u = bf16(x Wu^T); h = SiLU(g) * u, s = SiLU(g), u stored,
// codes of g; g stored when non-null. Same requirements as launch_linear_act_fwd.
hipError_t launch_linear_glu_fwd(int64_t M, int64_t N, int64_t K, const void* x, const void* w_gate,
                                 const void* w_up, void* h, void* s_out, void* u, uint32_t* codes,
                                 void* g, hipStream_t s);

// The same layers with MS-RMSNorm in front (Sec. 5.2 eq. norm_linear): x [M x K] is the
// norm's input. A statistics pre-pass writes rstd (fp32, per row, the norm kernel's
// arithmetic); the GEMM runs on x, scales each row's fp32 sums by its rstd before the
// bias, and its blocks store the norm's output z_norm = bf16(x rstd) [M x K] after their
// K loops. pre / g: the rounded pre-activation (gate), stored when non-null. x, w,
// z_norm 16-byte aligned; K % 8 == 0, N % 16 == 0.
hipError_t launch_linear_rms_act_fwd(int act, int64_t M, int64_t N, int64_t K, float eps,
                                     const void* x, const void* w, const void* bias, void* y,
                                     uint32_t* codes, void* pre, void* z_norm, float* rstd,
                                     hipStream_t s);
hipError_t launch_linear_rms_glu_fwd(int64_t M, int64_t N, int64_t K, float eps, const void* x,
                                     const void* w_gate, const void* w_up, void* h, void* s_out,
                                     void* u, uint32_t* codes, void* g, void* z_norm, float* rstd,
                                     hipStream_t s);

hipError_t launch_copy(const void* src, void* dst, int64_t bytes, hipStream_t s);

}  // namespace lmbp
