"""Parity at the full workload sizes, in the launch configuration the benchmark
times (same entry points, preallocated outputs). Every element of every output is
compared with the oracle: the host works through the tensors in blocks of rows so
that its float64 copies stay small."""

import numpy as np
import pytest
import torch

import oracle
import paper_2406_16282_amd as lmbp
from paper_2406_16282_amd import inputs
from compare import assert_codes_equal, assert_mixed, assert_rel, rtol_for

pytestmark = pytest.mark.gpu
DEV = "cuda:0"

ACT = {"regelu2": (lmbp.regelu2_fwd, lmbp.regelu2_bwd, oracle.regelu2_fwd, oracle.GELU_A),
       "resilu2": (lmbp.resilu2_fwd, lmbp.resilu2_bwd, oracle.resilu2_fwd, oracle.SILU_A)}
NORM = {"msln": (lmbp.msln_fwd, lmbp.msln_bwd, oracle.msln_fwd, oracle.msln_bwd),
        "msrms": (lmbp.msrms_fwd, lmbp.msrms_bwd, oracle.msrms_fwd, oracle.msrms_bwd)}
FULL = ["llama7b_swiglu_bf16", "llama13b_outliers_bf16", "vit_b_bs64_bf16_x12", "vit_b_fp32"]
BLOCK_ELEMS = 8 << 20          # host block: about 8M elements (a multiple of whole rows)


def T(a):
    return inputs.storage_to_torch(a, DEV)


def H(t):
    return inputs.torch_to_storage(t)


def row_blocks(rows, cols):
    step = max(1, BLOCK_ELEMS // cols)
    for r0 in range(0, rows, step):
        yield r0, min(rows, r0 + step)


@pytest.mark.parametrize("name", FULL)
def test_activation_full_size(name):
    w = inputs.WORKLOADS[name]
    s = w.act
    fwd, bwd, ofwd, a = ACT[s.op]
    print(f"[full] {name}: {s.op} {s.dtype} [{s.rows}x{s.cols}]", flush=True)
    x = w.act_x().reshape(s.rows, s.cols)
    dy = w.act_dy().reshape(s.rows, s.cols)
    xt, dyt = T(x), T(dy)
    y = torch.empty_like(xt)
    codes = torch.empty(lmbp.codes_words(xt.numel()), dtype=torch.int32, device=DEV)
    dx = torch.empty_like(dyt)
    fwd(xt, y=y, codes=codes)
    torch.cuda.synchronize()
    # The backward consumes the oracle's codes, which the loop below also checks
    # against the forward's, block by block.
    y_h, codes_h = H(y), H(codes).view(np.uint32)
    w_blocks = []
    rtol = rtol_for(s.dtype)
    per_row = s.cols // 16              # every row starts a code word (cols % 16 == 0)
    for r0, r1 in row_blocks(s.rows, s.cols):
        y_o, w_o = ofwd(oracle.decode(x[r0:r1], s.dtype))
        assert_codes_equal(codes_h[r0 * per_row:r1 * per_row], w_o, f"{name} codes rows {r0}:{r1}")
        y64 = oracle.decode(y_h[r0:r1], s.dtype)
        assert_rel(y64, y_o, rtol, f"{name} y rows {r0}:{r1} (strict)")
        assert_mixed(y64, y_o, rtol, f"{name} y rows {r0}:{r1}")
        w_blocks.append(w_o)
    bwd(dyt, T(np.concatenate(w_blocks)), dx=dx)
    torch.cuda.synchronize()
    dx_h = H(dx)
    lv = oracle.derivative_levels(a)
    for (r0, r1), w_o in zip(row_blocks(s.rows, s.cols), w_blocks):
        c = oracle.unpack_codes(w_o, (r1 - r0) * s.cols).reshape(r1 - r0, s.cols)
        dx_o = oracle.decode(dy[r0:r1], s.dtype) * lv[c]
        assert_rel(oracle.decode(dx_h[r0:r1], s.dtype), dx_o, rtol, f"{name} dx rows {r0}:{r1}", floor=0.0)
    print(f"[full] {name}: all {s.rows * s.cols} elements compared", flush=True)


@pytest.mark.parametrize("name", FULL)
def test_norm_full_size(name):
    w = inputs.WORKLOADS[name]
    s = w.norm
    fwd, bwd, ofwd, obwd = NORM[s.op]
    print(f"[full] {name}: {s.op} {s.dtype} [{s.rows}x{s.cols}]", flush=True)
    eps = float(np.float32(s.eps))
    x = w.norm_x()
    dz = w.norm_dz()
    # oracle forward in blocks; its stored state (z in the storage format, fp32 rstd) is
    # what both backward passes consume
    z_saved = np.empty_like(x)
    r_o = np.empty(s.rows, dtype=np.float64)
    for r0, r1 in row_blocks(s.rows, s.cols):
        z_o, r_o[r0:r1] = ofwd(oracle.decode(x[r0:r1], s.dtype), eps)
        z_saved[r0:r1] = oracle.encode(z_o, s.dtype)
    r_saved = r_o.astype(np.float32)
    xt = T(x)
    z = torch.empty_like(xt)
    rstd = torch.empty(s.rows, dtype=torch.float32, device=DEV)
    fwd(xt, eps, z=z, rstd=rstd)
    dzt = T(dz)
    dx = torch.empty_like(dzt)
    bwd(dzt, T(z_saved), T(r_saved), dx=dx)
    torch.cuda.synchronize()
    rtol = rtol_for(s.dtype)
    assert_rel(H(rstd).astype(np.float64), r_o, 1e-5, f"{name} rstd (all rows)", floor=0.0)
    z_h, dx_h = H(z), H(dx)
    for r0, r1 in row_blocks(s.rows, s.cols):
        z_o, _ = ofwd(oracle.decode(x[r0:r1], s.dtype), eps)
        assert_mixed(oracle.decode(z_h[r0:r1], s.dtype), z_o, rtol, f"{name} z rows {r0}:{r1}")
        dx_o = obwd(oracle.decode(dz[r0:r1], s.dtype), oracle.decode(z_saved[r0:r1], s.dtype),
                    r_saved[r0:r1])
        assert_mixed(oracle.decode(dx_h[r0:r1], s.dtype), dx_o, rtol, f"{name} dx rows {r0}:{r1}")
    print(f"[full] {name}: all {s.rows} rows compared", flush=True)
