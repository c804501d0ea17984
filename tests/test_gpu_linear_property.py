"""Randomised exact parity of the fused linear layers (hypothesis, fixed seed): random
m, n (multiple of 16), k (multiple of 8), activation and bias on dyadic inputs, whose
fp32 accumulation is exact in any order, so z, u and codes compare bit for bit."""

import os

import numpy as np
import pytest
import torch
from hypothesis import HealthCheck, given, settings, strategies as st

import oracle
import paper_2406_16282_amd as lmbp
from paper_2406_16282_amd import inputs
from compare import assert_mixed, assert_rel

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
# LMBP_PROPERTY_EXAMPLES raises the number of cases; LMBP_PROPERTY_RANDOM=1 draws them afresh
# (the default is a fixed, derandomized set).
SETTINGS = settings(max_examples=int(os.environ.get("LMBP_PROPERTY_EXAMPLES", 25)), deadline=None,
                    derandomize=os.environ.get("LMBP_PROPERTY_RANDOM", "0") != "1", database=None,
                    suppress_health_check=[HealthCheck.too_slow])


def T(a):
    return inputs.storage_to_torch(a, DEV)


def H(t):
    return inputs.torch_to_storage(t)


@SETTINGS
@given(m=st.integers(1, 700), n16=st.integers(1, 40), k8=st.integers(1, 80),
       act=st.sampled_from(["gelu", "silu"]), bias=st.booleans(), seed=st.integers(0, 2 ** 16))
def test_linear_act_random(m, n16, k8, act, bias, seed):
    n, k = 16 * n16, 8 * k8
    x = inputs.dyadic((m, k), -3, seed=seed, tensor_id=inputs.LIN_X)
    w = inputs.dyadic((n, k), -4, seed=seed, tensor_id=inputs.LIN_W)
    b = inputs.dyadic((n,), -7, seed=seed, tensor_id=inputs.LIN_B) if bias else None
    y, codes, z = lmbp.linear_act_fwd(T(x), T(w), None if b is None else T(b), act=act, store_z=True)
    torch.cuda.synchronize()
    _, z_s, y_o, c_o = oracle.linear_act_fwd(x, w, b, act)
    assert np.array_equal(H(z), z_s)
    assert np.array_equal(H(codes), c_o)
    assert_rel(oracle.decode(H(y), "bf16"), y_o, 1e-2, "y (strict)")


@SETTINGS
@given(m=st.integers(1, 500), n16=st.integers(1, 24), k8=st.integers(1, 48),
       seed=st.integers(0, 2 ** 16))
def test_linear_swiglu_random(m, n16, k8, seed):
    n, k = 16 * n16, 8 * k8
    x = inputs.dyadic((m, k), -3, seed=seed, tensor_id=inputs.LIN_X)
    wg = inputs.dyadic((n, k), -4, seed=seed, tensor_id=inputs.LIN_W)
    wu = inputs.dyadic((n, k), -4, seed=seed, tensor_id=inputs.LIN_B)
    h, s, u, codes, g = lmbp.linear_swiglu_fwd(T(x), T(wg), T(wu), store_g=True)
    torch.cuda.synchronize()
    _, g_s, _, u_s, h_o, s_o, c_o = oracle.linear_swiglu_fwd(x, wg, wu)
    assert np.array_equal(H(g), g_s) and np.array_equal(H(u), u_s)
    assert np.array_equal(H(codes), c_o)
    assert_rel(oracle.decode(H(s), "bf16"), s_o, 1e-2, "s (strict)")
    assert_mixed(oracle.decode(H(h), "bf16").reshape(m, n), h_o, 1e-2, "h")
