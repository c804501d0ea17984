"""Parity at the full workload sizes, in the launch configuration the benchmark
times (same entry points, preallocated outputs). Codes are compared in full; float
outputs on a random sample of elements (activations) or rows (norms), which the
oracle computes one by one."""

import numpy as np
import pytest
import torch

import oracle
import paper_2406_16282_amd as lmbp
from paper_2406_16282_amd import inputs
from compare import assert_codes_equal, assert_mixed, assert_rel, rtol_for

pytestmark = pytest.mark.gpu
DEV = "cuda:0"

ACT = {"regelu2": (lmbp.regelu2_fwd, lmbp.regelu2_bwd, oracle.gelu, oracle.GELU_A, oracle.GELU_C),
       "resilu2": (lmbp.resilu2_fwd, lmbp.resilu2_bwd, oracle.silu, oracle.SILU_A, oracle.SILU_C)}
NORM = {"msln": (lmbp.msln_fwd, lmbp.msln_bwd, oracle.msln_fwd, oracle.msln_bwd),
        "msrms": (lmbp.msrms_fwd, lmbp.msrms_bwd, oracle.msrms_fwd, oracle.msrms_bwd)}
FULL = ["llama7b_swiglu_bf16", "llama13b_outliers_bf16", "vit_b_bs64_bf16_x12", "vit_b_fp32"]


def T(a):
    return inputs.storage_to_torch(a, DEV)


def H(t):
    return inputs.torch_to_storage(t)


@pytest.mark.parametrize("name", FULL)
def test_activation_full_size(name):
    w = inputs.WORKLOADS[name]
    s = w.act
    fwd, bwd, h, a, c = ACT[s.op]
    print(f"[full] {name}: {s.op} {s.dtype} [{s.rows}x{s.cols}]", flush=True)
    x = w.act_x()
    dy = w.act_dy()
    x64 = oracle.decode(x, s.dtype).reshape(-1)
    w_o = oracle.pack_codes(oracle.segment_code(x64, c))
    xt, dyt = T(x), T(dy)
    y = torch.empty_like(xt)
    codes = torch.empty(lmbp.codes_words(xt.numel()), dtype=torch.int32, device=DEV)
    dx = torch.empty_like(dyt)
    fwd(xt, y=y, codes=codes)
    bwd(dyt, T(w_o), dx=dx)
    torch.cuda.synchronize()
    assert_codes_equal(H(codes), w_o, f"{name} codes")
    idx = np.sort(np.random.default_rng(0).choice(x64.size, size=200_000, replace=False))
    rtol = rtol_for(s.dtype)
    y_s = oracle.decode(H(y).reshape(-1)[idx], s.dtype)
    assert_rel(y_s, h(x64[idx]), rtol, f"{name} y (sample)")
    codes_s = oracle.unpack_codes(w_o, x64.size)[idx]
    dx_ref = oracle.decode(dy.reshape(-1)[idx], s.dtype) * oracle.derivative_levels(a)[codes_s]
    assert_rel(oracle.decode(H(dx).reshape(-1)[idx], s.dtype), dx_ref, rtol, f"{name} dx (sample)", floor=0.0)


@pytest.mark.parametrize("name", FULL)
def test_norm_full_size(name):
    w = inputs.WORKLOADS[name]
    s = w.norm
    fwd, bwd, ofwd, obwd = NORM[s.op]
    print(f"[full] {name}: {s.op} {s.dtype} [{s.rows}x{s.cols}]", flush=True)
    eps = float(np.float32(s.eps))
    x = w.norm_x()
    dz = w.norm_dz()
    z_o, r_o = ofwd(oracle.decode(x, s.dtype), eps)
    z_saved = oracle.encode(z_o, s.dtype)
    r_saved = r_o.astype(np.float32)
    xt = T(x)
    z = torch.empty_like(xt)
    rstd = torch.empty(s.rows, dtype=torch.float32, device=DEV)
    fwd(xt, eps, z=z, rstd=rstd)
    dzt = T(dz)
    dx = torch.empty_like(dzt)
    bwd(dzt, T(z_saved), T(r_saved), dx=dx)
    torch.cuda.synchronize()
    rows = np.sort(np.random.default_rng(1).choice(s.rows, size=min(256, s.rows), replace=False))
    rtol = rtol_for(s.dtype)
    assert_rel(H(rstd).astype(np.float64), r_o, 1e-5, f"{name} rstd (all rows)", floor=0.0)
    assert_mixed(oracle.decode(H(z)[rows], s.dtype), z_o[rows], rtol, f"{name} z (rows)")
    dx_o = obwd(oracle.decode(dz[rows], s.dtype), oracle.decode(z_saved[rows], s.dtype), r_saved[rows])
    assert_mixed(oracle.decode(H(dx)[rows], s.dtype), dx_o, rtol, f"{name} dx (rows)")
