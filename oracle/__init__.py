"""Reference oracle for the Approx-BP / MS-BP hot path: plain, slow, fp64, CPU only.

TEST INFRASTRUCTURE. Only the test suite, the smoke check in ``__graft_entry__`` and
the CPU-baseline leg of ``bench.py`` may import this package. The product path
(the HIP library and its Python binding) never imports it, and it imports nothing
from the product path: no kernels, headers, helpers, tables or constants are shared.

What it computes, each function citing the passage it follows:

* ``activations``: ReGELU2 / ReSiLU2 (Sec. 4.2, eq. relus_family with k = 2;
  constants from Appendix E): exact GELU/SiLU forward, the 2-bit segment code of
  every element, LSB-first packing 16 codes per 32-bit word, and the backward pass
  ``dx = dy * (slope of the ReLU combination on the element's segment)``.
* ``activations`` also holds ReSiLU2 inside a SwiGLU product (h = SiLU(g) * u), the
  form it takes in the LLaMA MLP.
* ``variants``: the general k-bit family and Appendix I's ReGELU2-d constants.
* ``norms``: MS-LN and MS-RMSNorm (Sec. 5.2 Alg. 1; Appendix G Alg. 2 and Alg. 3):
  forward ``z = H x / sigma`` saving ``z`` and ``1/sigma``; backward
  ``dx = sigma^-1 (H - p^-1 z z^T) dz`` from the saved output alone.
* ``linear``: a linear layer z = x W^T + b whose output, rounded once to bf16, feeds
  ReGELU2 / ReSiLU2 (the fused forward of the MLP's first projection), and the gated
  form (two projections feeding ReSiLU2 inside SwiGLU); both also with MS-RMSNorm in
  front (the norm's output feeding the merged layer, Sec. 5.2 eq. norm_linear).
* ``dtypes``: decoding of fp32 / bf16 storage to fp64 and correct round-to-nearest-even
  encoding of fp64 results back to storage.

All arithmetic is float64. Every function is pinned by a CPU test against
something other than itself (library routines of other implementations, closed
forms, invariants, brute force, finite differences); see ``tests/test_oracle_*.py``.
"""

from .dtypes import decode, encode, round_to_dtype, DTYPES
from .activations import (
    GELU_A, GELU_C, SILU_A, SILU_C,
    relu_combination, derivative_levels, segment_code,
    gelu, silu, pack_codes, unpack_codes, codes_words,
    regelu2_fwd, regelu2_bwd, resilu2_fwd, resilu2_bwd,
    reswiglu2_fwd, reswiglu2_bwd,
)
from .norms import msln_fwd, msln_bwd, msrms_fwd, msrms_bwd
from . import variants
from .linear import (linear, linear_act_fwd, linear_swiglu_fwd, msrms_linear_act_fwd,
                     msrms_linear_swiglu_fwd)

__all__ = [
    "decode", "encode", "round_to_dtype", "DTYPES",
    "GELU_A", "GELU_C", "SILU_A", "SILU_C",
    "relu_combination", "derivative_levels", "segment_code",
    "gelu", "silu", "pack_codes", "unpack_codes", "codes_words",
    "regelu2_fwd", "regelu2_bwd", "resilu2_fwd", "resilu2_bwd",
    "reswiglu2_fwd", "reswiglu2_bwd",
    "msln_fwd", "msln_bwd", "msrms_fwd", "msrms_bwd", "variants",
    "linear", "linear_act_fwd", "linear_swiglu_fwd", "msrms_linear_act_fwd", "msrms_linear_swiglu_fwd",
]
