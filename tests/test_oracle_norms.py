"""Pins of the oracle's MS-LN / MS-RMSNorm (Sec. 5.2 Alg. 1, Appendix G Alg. 2 / Alg. 3)."""

import numpy as np
import pytest

import oracle
import pins

NORMS = {
    "ln": (oracle.msln_fwd, oracle.msln_bwd, True),
    "rms": (oracle.msrms_fwd, oracle.msrms_bwd, False),
}


def test_ln_forward_against_torch():
    assert pins.pin_ln_fwd_torch(oracle.msln_fwd) < 1e-12


def test_rms_forward_against_torch():
    assert pins.pin_rms_fwd_torch(oracle.msrms_fwd) < 1e-12


@pytest.mark.parametrize("kind", ["ln", "rms"])
@pytest.mark.parametrize("eps", [1e-6, 1e-5, 0.3])
def test_backward_against_finite_differences(kind, eps):
    fwd, bwd, _ = NORMS[kind]
    assert pins.pin_norm_fd(fwd, bwd, eps) < 1e-6


@pytest.mark.parametrize("kind", ["ln", "rms"])
def test_backward_against_torch_autograd(kind):
    fwd, bwd, centered = NORMS[kind]
    assert pins.pin_norm_autograd(fwd, bwd, centered, 1e-5) < 1e-12


@pytest.mark.parametrize("kind", ["ln", "rms"])
def test_affine_merge_equivalence(kind):
    fwd, bwd, centered = NORMS[kind]
    assert pins.pin_affine_merge(fwd, bwd, centered, 1e-6) < 1e-12


@pytest.mark.parametrize("kind", ["ln", "rms"])
@pytest.mark.parametrize("eps", [1e-6, 1e-2])
def test_invariants(kind, eps):
    fwd, bwd, centered = NORMS[kind]
    assert pins.pin_norm_invariants(fwd, bwd, centered, eps) < 1e-10


def test_degenerate_rows():
    eps = 1e-6
    x = np.full((2, 5), 3.0)
    z, rstd = oracle.msln_fwd(x, eps)
    assert np.all(z == 0.0) and np.allclose(rstd, eps ** -0.5, rtol=1e-15)
    dx = oracle.msln_bwd(np.random.default_rng(0).normal(size=x.shape), z, rstd)
    # constant row: z = 0, so dx = rstd * (dz - mean dz)
    assert np.all(np.isfinite(dx))
    z1, r1 = oracle.msln_fwd(np.array([[7.0], [-2.0]]), eps)
    assert np.all(z1 == 0.0)
    zr, rr = oracle.msrms_fwd(np.zeros((1, 4)), 1e-5)
    assert np.all(zr == 0.0) and rr[0] == pytest.approx(1e-5 ** -0.5, rel=1e-15)
    dz = np.array([[1.0, -2.0, 3.0, 0.5]])
    assert np.allclose(oracle.msrms_bwd(dz, zr, rr), rr[0] * dz, rtol=1e-15)
