"""Pins of the oracle's fused ReSiLU2-SwiGLU (h = SiLU(g) * u with the ReSiLU2 backward)."""

import numpy as np
import pytest

import oracle
import pins


def test_backward_against_finite_differences():
    assert pins.pin_swiglu_fd(oracle.reswiglu2_fwd, oracle.reswiglu2_bwd, oracle.relu_combination,
                              oracle.SILU_A, oracle.SILU_C) < 1e-6


def test_reduces_to_resilu2_when_u_is_one():
    assert pins.pin_swiglu_reduces_to_resilu2(oracle.reswiglu2_fwd, oracle.reswiglu2_bwd,
                                              oracle.resilu2_fwd, oracle.resilu2_bwd) < 1e-15


def test_forward_against_torch():
    import torch
    import torch.nn.functional as F
    g = np.linspace(-20, 20, 801)
    u = np.cos(g)
    h, s, _ = oracle.reswiglu2_fwd(g, u)
    ref = (F.silu(torch.from_numpy(g)) * torch.from_numpy(u)).numpy()
    assert np.max(np.abs(h - ref) / np.maximum(np.abs(ref), 1e-300)) < 1e-14


def test_shape_mismatch_rejected():
    with pytest.raises(ValueError):
        oracle.reswiglu2_fwd(np.zeros(3), np.zeros(4))
