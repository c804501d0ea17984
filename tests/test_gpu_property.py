"""Randomised parity (hypothesis, fixed seed): random shapes, dtypes, ops and base
offsets through the C ABI against the oracle, plus the plain-copy utility."""

import os

import numpy as np
import pytest
import torch
from hypothesis import HealthCheck, given, settings, strategies as st

import oracle
import paper_2406_16282_amd as lmbp
from paper_2406_16282_amd import inputs
from compare import assert_codes_equal, assert_mixed, assert_rel, norm_grad_scale, rtol_for

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
# LMBP_PROPERTY_EXAMPLES raises the number of cases; LMBP_PROPERTY_RANDOM=1 draws them afresh
# (the default is a fixed, derandomized set).
SETTINGS = settings(max_examples=int(os.environ.get("LMBP_PROPERTY_EXAMPLES", 40)), deadline=None,
                    derandomize=os.environ.get("LMBP_PROPERTY_RANDOM", "0") != "1", database=None,
                    suppress_health_check=[HealthCheck.too_slow])


def T(a):
    return inputs.storage_to_torch(a, DEV)


def H(t):
    return inputs.torch_to_storage(t)


def on_device(arr, offset):
    """Device tensor holding ``arr`` starting ``offset`` elements into an allocation."""
    flat = arr.reshape(-1)
    pad = np.concatenate([flat[:1].repeat(offset), flat]) if offset else flat
    return T(pad)[offset:].view(arr.shape)


@SETTINGS
@given(op=st.sampled_from(["regelu2", "resilu2"]), dtype=st.sampled_from(["fp32", "bf16"]),
       n=st.integers(1, 70_000), offset=st.integers(0, 3), std=st.sampled_from([0.5, 2.0, 8.0]),
       seed=st.integers(0, 2 ** 16))
def test_activation_random(op, dtype, n, offset, std, seed):
    fwd, bwd = (lmbp.regelu2_fwd, lmbp.regelu2_bwd) if op == "regelu2" else (lmbp.resilu2_fwd, lmbp.resilu2_bwd)
    ofwd, obwd = (oracle.regelu2_fwd, oracle.regelu2_bwd) if op == "regelu2" else (oracle.resilu2_fwd, oracle.resilu2_bwd)
    x = inputs.normal((n,), std, dtype, seed=seed, tensor_id=inputs.ACT_X)
    dy = inputs.normal((n,), 1.0, dtype, seed=seed, tensor_id=inputs.ACT_DY)
    y, codes = fwd(on_device(x, offset))
    y_o, w_o = ofwd(oracle.decode(x, dtype))
    dx = bwd(on_device(dy, offset), T(w_o))
    torch.cuda.synchronize()
    assert_codes_equal(H(codes), w_o, "codes")
    rtol = rtol_for(dtype)
    assert_rel(oracle.decode(H(y), dtype), y_o, rtol, "y")
    assert_rel(oracle.decode(H(dx), dtype), obwd(oracle.decode(dy, dtype), w_o), rtol, "dx", floor=0.0)


@SETTINGS
@given(op=st.sampled_from(["msln", "msrms"]), dtype=st.sampled_from(["fp32", "bf16"]),
       rows=st.integers(1, 40), cols=st.integers(1, 9000), offset=st.integers(0, 1),
       seed=st.integers(0, 2 ** 16))
def test_norm_random(op, dtype, rows, cols, offset, seed):
    fwd, bwd = (lmbp.msln_fwd, lmbp.msln_bwd) if op == "msln" else (lmbp.msrms_fwd, lmbp.msrms_bwd)
    ofwd, obwd = (oracle.msln_fwd, oracle.msln_bwd) if op == "msln" else (oracle.msrms_fwd, oracle.msrms_bwd)
    eps = float(np.float32(1e-5))
    x = inputs.normal((rows, cols), 1.0, dtype, seed=seed, tensor_id=inputs.NORM_X, mean=0.5)
    dz = inputs.normal((rows, cols), 1.0, dtype, seed=seed, tensor_id=inputs.NORM_DZ)
    z_o, r_o = ofwd(oracle.decode(x, dtype), eps)
    z_s = oracle.encode(z_o, dtype)
    dx_o = obwd(oracle.decode(dz, dtype), oracle.decode(z_s, dtype), r_o.astype(np.float32))
    z, rstd = fwd(on_device(x, offset), eps)
    dx = bwd(on_device(dz, offset), on_device(z_s, offset), T(r_o.astype(np.float32)))
    torch.cuda.synchronize()
    rtol = rtol_for(dtype)
    assert_mixed(oracle.decode(H(z), dtype), z_o, rtol, "z")
    assert_rel(H(rstd).astype(np.float64), r_o, 1e-5, "rstd", floor=0.0)
    assert_mixed(oracle.decode(H(dx), dtype), dx_o, rtol, "dx",
                 row_scale=norm_grad_scale(oracle.decode(dz, dtype), r_o.astype(np.float32)))


@SETTINGS
@given(dtype=st.sampled_from(["fp32", "bf16"]), n=st.integers(1, 70_000), offset=st.integers(0, 3),
       seed=st.integers(0, 2 ** 16))
def test_swiglu_random(dtype, n, offset, seed):
    g = inputs.normal((n,), 2.0, dtype, seed=seed, tensor_id=inputs.ACT_X)
    u = inputs.normal((n,), 1.0, dtype, seed=seed, tensor_id=inputs.ACT_U)
    dh = inputs.normal((n,), 1.0, dtype, seed=seed, tensor_id=inputs.ACT_DY)
    h, s, codes = lmbp.reswiglu2_fwd(on_device(g, offset), on_device(u, offset))
    h_o, s_o, w_o = oracle.reswiglu2_fwd(oracle.decode(g, dtype), oracle.decode(u, dtype))
    s_saved = oracle.encode(s_o, dtype)
    dg, du = lmbp.reswiglu2_bwd(on_device(dh, offset), on_device(u, offset), on_device(s_saved, offset),
                                T(w_o))
    dg_o, du_o = oracle.reswiglu2_bwd(oracle.decode(dh, dtype), oracle.decode(u, dtype),
                                      oracle.decode(s_saved, dtype), w_o)
    torch.cuda.synchronize()
    assert_codes_equal(H(codes), w_o, "codes")
    rtol = rtol_for(dtype)
    assert_rel(oracle.decode(H(s), dtype), s_o, rtol, "s")
    assert_rel(oracle.decode(H(h), dtype), h_o, rtol, "h")
    assert_rel(oracle.decode(H(dg), dtype), dg_o, rtol, "dg")
    assert_rel(oracle.decode(H(du), dtype), du_o, rtol, "du")


@SETTINGS
@given(bits=st.sampled_from([1, 2, 3, 4]), act=st.sampled_from(["gelu", "silu"]),
       dtype=st.sampled_from(["fp32", "bf16"]), n=st.integers(1, 30_000), offset=st.integers(0, 3),
       seed=st.integers(0, 2 ** 16))
def test_stepact_random(bits, act, dtype, n, offset, seed):
    from oracle import variants as OV
    r = np.random.default_rng(seed)
    m = (1 << bits) - 1
    c = list(np.sort(r.uniform(-5, 5, m)) + np.arange(m) * 1e-3)
    lv = list(r.normal(0, 0.5, m + 1))
    x = inputs.normal((n,), 3.0, dtype, seed=seed, tensor_id=inputs.ACT_X)
    dy = inputs.normal((n,), 1.0, dtype, seed=seed, tensor_id=inputs.ACT_DY)
    y, codes = lmbp.stepact_fwd(on_device(x, offset), act, c, bits)
    y_o, w_o = OV.stepact_fwd(oracle.decode(x, dtype), act, c, bits)
    dx = lmbp.stepact_bwd(on_device(dy, offset), T(w_o), lv, bits)
    lv32 = np.asarray(lv, dtype=np.float32).astype(np.float64)
    dx_o = OV.stepact_bwd(oracle.decode(dy, dtype), w_o, lv32, bits)
    torch.cuda.synchronize()
    assert_codes_equal(H(codes), w_o, "codes")
    rtol = rtol_for(dtype)
    assert_rel(oracle.decode(H(y), dtype), y_o, rtol, "y")
    assert_rel(oracle.decode(H(dx), dtype), dx_o, rtol, "dx", floor=0.0)


@pytest.mark.parametrize("nbytes", [1, 15, 16, 17, 4096, 4096 * 257 + 9, 3 * 2 ** 20 + 5])
def test_copy_utility(nbytes):
    src = torch.randint(0, 256, (nbytes,), dtype=torch.uint8, device=DEV)
    dst = torch.zeros_like(src)
    lmbp.copy_bytes(src, dst)
    torch.cuda.synchronize()
    assert torch.equal(src, dst)
