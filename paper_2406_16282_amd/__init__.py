"""lmbp: MI355X (gfx950) HIP kernels for the hot path of Approximate and
Memory-Sharing Backpropagation (Yang et al., ICML 2024).

ReGELU2 / ReSiLU2 keep the exact activation in the forward pass and save only a
2-bit segment code per element for a step-function derivative in the backward
pass (Sec. 4.2); ReSiLU2 also comes fused with the SwiGLU product of the LLaMA
MLP, and both come fused into the epilogue of the preceding linear layer's matrix
product (bf16 MFMA). MS-LN / MS-RMSNorm, with the affine merged into the next
linear layer, save only their output and one fp32 statistic per row (Sec. 5.2);
MS-RMSNorm also comes fused into that linear layer's matrix product.

The kernels live in liblmbp.so (C ABI in include/lmbp.h); ``binding`` marshals
torch tensors into it. The library is loaded on first use.
"""

from .binding import (  # noqa: F401
    LmbpError,
    codes_bytes,
    codes_words,
    copy_bytes,
    lib,
    linear_act_fwd,
    linear_swiglu_fwd,
    msln_bwd,
    msln_fwd,
    msrms_bwd,
    msrms_fwd,
    msrms_linear_act_fwd,
    msrms_linear_swiglu_fwd,
    regelu2_bwd,
    regelu2_fwd,
    resilu2_bwd,
    resilu2_fwd,
    reswiglu2_bwd,
    reswiglu2_fwd,
    stepact_bwd,
    stepact_fwd,
)
