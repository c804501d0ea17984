"""Maximum sizes: tensors of more than 2^31 elements, so every index path must be 64-bit.

Inputs are the closed-form hash pattern of ``inputs.hash_tensor`` (built on the GPU); the
oracle recomputes the same values on the host for the sampled indices it checks: the
elements around index 2^31, the ragged tail, and random positions."""

import gc

import numpy as np
import pytest
import torch

import oracle
import paper_2406_16282_amd as lmbp
from paper_2406_16282_amd import inputs
from compare import assert_mixed, assert_rel

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
BIG = (1 << 31) + 4099          # not a multiple of 16: the last code word is partial


def H(t):
    return inputs.torch_to_storage(t)


def sample(n, extra=()):
    r = np.random.default_rng(0)
    idx = np.concatenate([r.integers(0, n, 200_000), np.arange((1 << 31) - 40, (1 << 31) + 40),
                          np.arange(n - 40, n), np.array(extra, dtype=np.int64)])
    return np.unique(idx[(idx >= 0) & (idx < n)])


@pytest.fixture(autouse=True)
def _free():
    yield
    gc.collect()
    torch.cuda.empty_cache()


@pytest.mark.parametrize("offset", [0, 1])
def test_resilu2_beyond_int32(offset):
    """offset 0: vector path; offset 1 (tensors one element past a 16-byte boundary):
    general path."""
    print(f"[large] resilu2 bf16 n={BIG} offset={offset}", flush=True)
    n = BIG - offset
    xfull = inputs.hash_tensor(BIG, "bf16", DEV)
    x = xfull[offset:]
    y, codes = lmbp.resilu2_fwd(x)
    del xfull, x
    dyfull = inputs.hash_tensor(BIG, "bf16", DEV, scale=1.0, salt=977)
    dy = dyfull[offset:]
    dx = lmbp.resilu2_bwd(dy, codes)
    torch.cuda.synchronize()
    idx = sample(n)
    it = torch.from_numpy(idx).to(DEV)
    y_s = H(y[it])
    dx_s = H(dx[it])
    words = H(codes[torch.from_numpy(np.unique(idx // 16)).to(DEV)])
    x64 = oracle.decode(inputs.hash_storage(idx + offset, "bf16"), "bf16")
    dy64 = oracle.decode(inputs.hash_storage(idx + offset, "bf16", scale=1.0, salt=977), "bf16")
    code_o = oracle.segment_code(x64, oracle.SILU_C)
    wpos = np.searchsorted(np.unique(idx // 16), idx // 16)
    code_g = (words.astype(np.uint64)[wpos] >> (2 * (idx % 16)).astype(np.uint64)) & 3
    assert np.array_equal(code_g.astype(np.uint8), code_o), "codes differ beyond 2^31"
    # the unused bits of the last word are zero
    last = int(H(codes[-1:])[0])
    used = n % 16
    assert used == 0 or last >> (2 * used) == 0
    assert_rel(oracle.decode(y_s, "bf16"), oracle.silu(x64), 1e-2, "y beyond 2^31")
    lv = oracle.derivative_levels(oracle.SILU_A)[code_o]
    assert_rel(oracle.decode(dx_s, "bf16"), dy64 * lv, 1e-2, "dx beyond 2^31", floor=0.0)


@pytest.mark.parametrize("op,cols", [("msrms", 4096), ("msln", 4100)])
def test_norm_beyond_int32(op, cols):
    """msrms with 4096-wide rows: register-tile path; msln with 4100-wide bf16 rows (not
    16-byte multiples): block-per-row path. Chained check: each side runs its own
    forward, then its backward."""
    rows = (1 << 31) // cols + 5
    n = rows * cols
    print(f"[large] {op} bf16 rows={rows} cols={cols} n={n}", flush=True)
    fwd, bwd = (lmbp.msrms_fwd, lmbp.msrms_bwd) if op == "msrms" else (lmbp.msln_fwd, lmbp.msln_bwd)
    ofwd, obwd = (oracle.msrms_fwd, oracle.msrms_bwd) if op == "msrms" else (oracle.msln_fwd, oracle.msln_bwd)
    eps = float(np.float32(1e-5))
    x = inputs.hash_tensor(n, "bf16", DEV).view(rows, cols)
    z, rstd = fwd(x, eps)
    del x
    dz = inputs.hash_tensor(n, "bf16", DEV, scale=1.0, salt=977).view(rows, cols)
    dx = bwd(dz, z, rstd)
    torch.cuda.synchronize()
    r = np.random.default_rng(1)
    sel = np.unique(np.concatenate([r.integers(0, rows, 64), [(1 << 31) // cols - 1, (1 << 31) // cols,
                                                             (1 << 31) // cols + 1, rows - 1]]))
    st = torch.from_numpy(sel).to(DEV)
    idx = (sel[:, None] * cols + np.arange(cols)[None, :])
    x64 = oracle.decode(inputs.hash_storage(idx, "bf16"), "bf16")
    dz64 = oracle.decode(inputs.hash_storage(idx, "bf16", scale=1.0, salt=977), "bf16")
    z_o, r_o = ofwd(x64, eps)
    # chained: the oracle's backward sees its own stored forward state (z rounded to
    # bf16, rstd to fp32), as the GPU's sees its own
    dx_o = obwd(dz64, oracle.round_to_dtype(z_o, "bf16"), r_o.astype(np.float32))
    assert_mixed(oracle.decode(H(z[st]), "bf16"), z_o, 1e-2, f"{op} z beyond 2^31")
    assert_rel(H(rstd[st]).astype(np.float64), r_o, 1e-5, f"{op} rstd beyond 2^31", floor=0.0)
    assert_mixed(oracle.decode(H(dx[st]), "bf16"), dx_o, 1e-2, f"{op} dx beyond 2^31 (chained)")
