"""A linear layer whose output feeds ReGELU2 / ReSiLU2 (Sec. 4.2), and the same with
MS-RMSNorm in front (Sec. 5.2 eq. norm_linear).

Test infrastructure only (see the package docstring).

The activation's input is the output z = x W^T + b of the preceding linear layer
(the MLP's first projection in ViT and LLaMA blocks). The fused GPU operation rounds
z once to bf16 and applies the activation to the rounded value, so that its y and
codes are those the stand-alone activation would produce from a stored bf16 z. The
oracle writes that composition out: the exact product in float64, the one rounding,
then the activation oracle of ``activations``.
"""

import numpy as np

from .activations import regelu2_fwd, resilu2_fwd, reswiglu2_fwd
from .dtypes import decode, encode
from .norms import msrms_fwd


def linear(x, w, b=None):
    """z = x W^T + b in float64 (x [m, k], w [n, k] as an nn.Linear weight, b [n])."""
    x = np.asarray(x, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    z = x @ w.T
    if b is not None:
        z = z + np.asarray(b, dtype=np.float64)[None, :]
    return z


def linear_act_fwd(x_bf16, w_bf16, b_bf16, act):
    """The fused forward on bf16 storage: returns (z exact, z stored as bf16 bits,
    y in float64 (the activation of the stored z), packed codes of the stored z)."""
    z = linear(decode(x_bf16, "bf16"), decode(w_bf16, "bf16"),
               None if b_bf16 is None else decode(b_bf16, "bf16"))
    z_s = encode(z, "bf16")
    fwd = {"gelu": regelu2_fwd, "silu": resilu2_fwd}[act]
    y, codes = fwd(decode(z_s, "bf16"))
    return z, z_s, y, codes


def linear_swiglu_fwd(x_bf16, wg_bf16, wu_bf16):
    """The gated form (the LLaMA MLP's input side, Sec. 6): g = x Wg^T and u = x Wu^T,
    each rounded once to bf16, then ReSiLU2 inside SwiGLU on the stored g and u.
    Returns (g exact, g stored, u exact, u stored, h and s in float64, packed codes of g)."""
    xd = decode(x_bf16, "bf16")
    g = linear(xd, decode(wg_bf16, "bf16"))
    u = linear(xd, decode(wu_bf16, "bf16"))
    g_s, u_s = encode(g, "bf16"), encode(u, "bf16")
    h, s, codes = reswiglu2_fwd(decode(g_s, "bf16"), decode(u_s, "bf16"))
    return g, g_s, u, u_s, h, s, codes


# ------------------------------------------------ MS-RMSNorm in front of the layer

def msrms_linear_act_fwd(x_bf16, w_bf16, b_bf16, act, eps):
    """MS-RMSNorm followed by the merged linear layer and ReGELU2 / ReSiLU2 (Sec. 5.2
    eq. norm_linear: y = W~ z + b~ with z the normalised row; App. G Alg. 3 for z).

    The norm's output enters the linear layer as computed (float64, before any storage
    rounding): the pre-activation is z W^T + b, rounded once to bf16, then the
    activation oracle. z is also returned rounded to bf16 (the saved tensor), and rstd.
    Returns (pre-activation exact, pre-activation stored, y in float64, packed codes,
    z stored as bf16 bits, rstd)."""
    z, rstd = msrms_fwd(decode(x_bf16, "bf16"), eps)
    p = linear(z, decode(w_bf16, "bf16"), None if b_bf16 is None else decode(b_bf16, "bf16"))
    p_s = encode(p, "bf16")
    fwd = {"gelu": regelu2_fwd, "silu": resilu2_fwd}[act]
    y, codes = fwd(decode(p_s, "bf16"))
    return p, p_s, y, codes, encode(z, "bf16"), rstd


def msrms_linear_swiglu_fwd(x_bf16, wg_bf16, wu_bf16, eps):
    """The gated form: MS-RMSNorm, then g = z Wg^T and u = z Wu^T (z as computed, each
    product rounded once to bf16), then ReSiLU2 inside SwiGLU on the stored g and u.
    Returns (g exact, g stored, u exact, u stored, h and s in float64, packed codes of g,
    z stored as bf16 bits, rstd)."""
    z, rstd = msrms_fwd(decode(x_bf16, "bf16"), eps)
    g = linear(z, decode(wg_bf16, "bf16"))
    u = linear(z, decode(wu_bf16, "bf16"))
    g_s, u_s = encode(g, "bf16"), encode(u, "bf16")
    h, s, codes = reswiglu2_fwd(decode(g_s, "bf16"), decode(u_s, "bf16"))
    return g, g_s, u, u_s, h, s, codes, encode(z, "bf16"), rstd
