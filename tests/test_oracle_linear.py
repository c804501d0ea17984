"""Pins of the linear-layer oracle (CPU): brute force, identity weights, exact
dyadic arithmetic, and the composition with the activation oracle."""

import math
from fractions import Fraction

import numpy as np
import pytest

import oracle
from paper_2406_16282_amd import inputs


def brute_linear(x, w, b):
    m, k = x.shape
    n = w.shape[0]
    out = np.empty((m, n))
    for i in range(m):
        for j in range(n):
            out[i, j] = math.fsum([x[i, t] * w[j, t] for t in range(k)] + ([b[j]] if b is not None else []))
    return out


@pytest.mark.parametrize("m,n,k", [(1, 1, 1), (3, 5, 4), (7, 2, 9), (4, 16, 8)])
def test_linear_brute_force(m, n, k):
    g = np.random.default_rng(m * 100 + n * 10 + k)
    x, w, b = g.standard_normal((m, k)), g.standard_normal((n, k)), g.standard_normal(n)
    np.testing.assert_allclose(oracle.linear(x, w, b), brute_linear(x, w, b), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(oracle.linear(x, w), brute_linear(x, w, None), rtol=1e-12, atol=1e-12)


def test_linear_identity_weight():
    g = np.random.default_rng(1)
    x, b = g.standard_normal((6, 5)), g.standard_normal(5)
    assert np.array_equal(oracle.linear(x, np.eye(5), b), x + b[None, :])


def test_linear_dyadic_is_exact():
    """Dyadic bf16 inputs: the float64 product equals the exact rational result."""
    x = inputs.dyadic((5, 24), -3, tensor_id=inputs.LIN_X)
    w = inputs.dyadic((7, 24), -4, tensor_id=inputs.LIN_W)
    b = inputs.dyadic((7,), -7, tensor_id=inputs.LIN_B)
    xd, wd, bd = (oracle.decode(a, "bf16") for a in (x, w, b))
    z = oracle.linear(xd, wd, bd)
    for i in range(5):
        for j in range(7):
            exact = sum(Fraction(xd[i, t]) * Fraction(wd[j, t]) for t in range(24)) + Fraction(bd[j])
            assert Fraction(z[i, j]) == exact


def test_linear_act_composition():
    """W = I, b = 0: the stored z is x itself and y, codes are the activation oracle's."""
    x = inputs.normal((4, 32), 2.0, "bf16", tensor_id=inputs.LIN_X)
    w = inputs.to_storage(np.eye(32), "bf16")
    for act, fwd in (("gelu", oracle.regelu2_fwd), ("silu", oracle.resilu2_fwd)):
        z, z_s, y, codes = oracle.linear_act_fwd(x, w, None, act)
        assert np.array_equal(z_s, x)
        y_ref, c_ref = fwd(oracle.decode(x, "bf16"))
        assert np.array_equal(codes, c_ref)
        assert np.array_equal(y, y_ref)


def test_linear_act_rounds_z_once():
    """z is rounded to bf16 once, to nearest even, before the activation."""
    x = inputs.to_storage(np.array([[1.0, 1.0]]), "bf16")
    # The bf16 step at 1 is 2^-7: 1 + 2^-8 is the midpoint and rounds to even (1.0),
    # 1 + 2^-8 + 2^-10 rounds up to 1 + 2^-7.
    w = inputs.to_storage(np.array([[1.0, 2.0 ** -8], [1.0, 2.0 ** -8 + 2.0 ** -10]]), "bf16")
    z, z_s, _, _ = oracle.linear_act_fwd(x, w, None, "gelu")
    assert z[0, 0] == 1.0 + 2.0 ** -8 and oracle.decode(z_s, "bf16")[0, 0] == 1.0
    assert oracle.decode(z_s, "bf16")[0, 1] == 1.0 + 2.0 ** -7


def test_linear_swiglu_composition():
    """Wg = Wu = I: g = u = x, and the outputs are the SwiGLU activation oracle's on (x, x)."""
    x = inputs.normal((4, 32), 2.0, "bf16", tensor_id=inputs.LIN_X)
    eye = inputs.to_storage(np.eye(32), "bf16")
    g, g_s, u, u_s, h, s, codes = oracle.linear_swiglu_fwd(x, eye, eye)
    assert np.array_equal(g_s, x) and np.array_equal(u_s, x)
    h_ref, s_ref, c_ref = oracle.reswiglu2_fwd(oracle.decode(x, "bf16"), oracle.decode(x, "bf16"))
    assert np.array_equal(h, h_ref) and np.array_equal(s, s_ref) and np.array_equal(codes, c_ref)


# ------------------------------------------------ MS-RMSNorm in front of the layer

def _torch_rms_then_linear(x, alpha, w, b, eps):
    """RMSNorm with affine alpha, then Linear(w, b), in float64 torch."""
    import torch
    import torch.nn.functional as F
    xt = torch.from_numpy(x)
    z = F.rms_norm(xt, (x.shape[1],), weight=torch.from_numpy(alpha), eps=eps)
    return F.linear(z, torch.from_numpy(w), None if b is None else torch.from_numpy(b)).numpy()


@pytest.mark.parametrize("act", ["gelu", "silu"])
def test_msrms_linear_against_torch_with_merged_affine(act):
    """RMSNorm(alpha) then Linear(W, b) (torch float64) equals the oracle's MS-RMSNorm in
    front of the merged layer W~ = W diag(alpha) (Sec. 5.2 eq. norm_linear). alpha holds
    powers of two so that W~ is exactly representable in bf16, as the stored weight is."""
    g = np.random.default_rng(21)
    m, k, n = 6, 64, 48
    eps = 1e-5
    x = inputs.normal((m, k), 1.5, "bf16", tensor_id=inputs.NORM_X)
    w = inputs.normal((n, k), 0.2, "bf16", tensor_id=inputs.LIN_W)
    b = inputs.normal((n,), 0.1, "bf16", tensor_id=inputs.LIN_B)
    alpha = 2.0 ** g.integers(-2, 3, k).astype(np.float64)
    wd = oracle.decode(w, "bf16")
    w_merged = inputs.to_storage(wd * alpha[None, :], "bf16")
    assert np.array_equal(oracle.decode(w_merged, "bf16"), wd * alpha[None, :])
    p, p_s, y, codes, z_s, rstd = oracle.msrms_linear_act_fwd(x, w_merged, b, act, eps)
    ref = _torch_rms_then_linear(oracle.decode(x, "bf16"), alpha, wd, oracle.decode(b, "bf16"), eps)
    np.testing.assert_allclose(p, ref, rtol=1e-12, atol=1e-12)
    # the stored z and rstd are the stand-alone norm's; y and codes the activation's of p_s
    z_o, r_o = oracle.msrms_fwd(oracle.decode(x, "bf16"), eps)
    assert np.array_equal(z_s, oracle.encode(z_o, "bf16")) and np.array_equal(rstd, r_o)
    fwd = oracle.regelu2_fwd if act == "gelu" else oracle.resilu2_fwd
    y_ref, c_ref = fwd(oracle.decode(p_s, "bf16"))
    assert np.array_equal(y, y_ref) and np.array_equal(codes, c_ref)


def test_msrms_linear_swiglu_against_torch():
    g = np.random.default_rng(22)
    m, k, n = 5, 40, 32
    eps = 1e-5
    x = inputs.normal((m, k), 1.0, "bf16", tensor_id=inputs.NORM_X)
    wg = inputs.normal((n, k), 0.3, "bf16", tensor_id=inputs.LIN_W)
    wu = inputs.normal((n, k), 0.3, "bf16", tensor_id=inputs.LIN_B)
    ones = np.ones(k)
    gx, g_s, ux, u_s, h, s, codes, z_s, rstd = oracle.msrms_linear_swiglu_fwd(x, wg, wu, eps)
    xd = oracle.decode(x, "bf16")
    np.testing.assert_allclose(gx, _torch_rms_then_linear(xd, ones, oracle.decode(wg, "bf16"), None, eps),
                               rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(ux, _torch_rms_then_linear(xd, ones, oracle.decode(wu, "bf16"), None, eps),
                               rtol=1e-12, atol=1e-12)
    h_ref, s_ref, c_ref = oracle.reswiglu2_fwd(oracle.decode(g_s, "bf16"), oracle.decode(u_s, "bf16"))
    assert np.array_equal(h, h_ref) and np.array_equal(s, s_ref) and np.array_equal(codes, c_ref)


def test_msrms_linear_uses_the_unrounded_norm_output():
    """The pre-activation is taken from z as computed, not from its bf16 storage: with a
    row whose z is not representable in bf16, the two differ and the oracle follows the
    former."""
    x = inputs.to_storage(np.array([[3.0, 1.0, 1.0, 1.0, 1.0, 1.0, 1.0, 1.0]]), "bf16")
    w = inputs.to_storage(np.eye(8)[:1].repeat(16, axis=0), "bf16")   # picks z[0], 16 outputs
    eps = float(np.float32(1e-5))
    p, p_s, _, _, z_s, rstd = oracle.msrms_linear_act_fwd(x, w, None, "silu", eps)
    z_exact = 3.0 / np.sqrt((9.0 + 7.0) / 8.0 + eps)
    assert np.allclose(p, z_exact, rtol=1e-14, atol=0)
    assert oracle.decode(z_s, "bf16")[0, 0] != z_exact
