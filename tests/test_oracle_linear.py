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
