"""GPU parity of MS-LN / MS-RMSNorm against the CPU oracle, through the C ABI.

The forward is compared directly. Both backward implementations consume the same
saved state: the oracle's z rounded to the storage dtype and its rstd rounded to
fp32."""

import numpy as np
import pytest
import torch

import oracle
import paper_2406_16282_amd as lmbp
from paper_2406_16282_amd import inputs
from compare import assert_mixed, assert_rel, norm_grad_scale, rtol_for

pytestmark = pytest.mark.gpu

NORMS = {
    "msln": (lmbp.msln_fwd, lmbp.msln_bwd, oracle.msln_fwd, oracle.msln_bwd),
    "msrms": (lmbp.msrms_fwd, lmbp.msrms_bwd, oracle.msrms_fwd, oracle.msrms_bwd),
}
DEV = "cuda:0"


def T(a):
    return inputs.storage_to_torch(a, DEV)


def H(t):
    return inputs.torch_to_storage(t)


def check_norm(op, dtype, x, dz, eps, label):
    fwd, bwd, ofwd, obwd = NORMS[op]
    print(f"[norm] {label}: op={op} dtype={dtype} shape={x.shape} eps={eps}", flush=True)
    rtol = rtol_for(dtype)
    eps32 = float(np.float32(eps))
    z_o, r_o = ofwd(oracle.decode(x, dtype), eps32)
    z_saved = oracle.encode(z_o, dtype)
    r_saved = r_o.astype(np.float32)
    dx_o = obwd(oracle.decode(dz, dtype), oracle.decode(z_saved, dtype), r_saved)

    z, rstd = fwd(T(x), eps32)
    dx = bwd(T(dz), T(z_saved), T(r_saved))
    torch.cuda.synchronize()

    assert_mixed(oracle.decode(H(z), dtype), z_o, rtol, f"{label} z")
    assert_rel(H(rstd).astype(np.float64), r_o, 1e-5, f"{label} rstd", floor=0.0)
    assert_mixed(oracle.decode(H(dx), dtype), dx_o, rtol, f"{label} dx",
                 row_scale=norm_grad_scale(oracle.decode(dz, dtype), r_saved))
    return z, rstd


CASES = [
    # (op, dtype, rows, cols, x_std, dz_std, eps)
    ("msln", "fp32", 8 * 197, 768, 1.0, 1.0, 1e-6),         # ViT-B fp32 block, full size
    ("msln", "bf16", 2048, 768, 1.5, 1e-2, 1e-6),           # ViT-B bf16 rows (subset)
    ("msrms", "bf16", 512, 4096, 1.0, 1e-3, 1e-5),          # LLaMA-7B rows (subset)
    ("msrms", "fp32", 256, 4096, 1.0, 1e-3, 1e-5),
    ("msln", "bf16", 5, 32768, 1.0, 1.0, 1e-6),             # widest register tile (bf16)
    ("msrms", "fp32", 5, 16384 + 4, 1.0, 1.0, 1e-5),        # just past the fp32 tile: block path
    ("msln", "bf16", 3, 32768 + 8, 1.0, 1.0, 1e-6),         # past the bf16 tile: block path
    ("msln", "fp32", 5, 1, 1.0, 1.0, 1e-6),                 # p = 1
    ("msrms", "bf16", 1, 8, 1.0, 1.0, 1e-5),                # one row, one vector
    ("msln", "fp32", 7, 72, 1.0, 1.0, 0.3),                 # large eps
    ("msrms", "bf16", 333, 5120, 1.0, 1e-3, 1e-5),          # LLaMA-13B width, rows not /4
]


@pytest.mark.parametrize("op,dtype,rows,cols,xs,gs,eps", CASES)
def test_parity(op, dtype, rows, cols, xs, gs, eps):
    x = inputs.normal((rows, cols), xs, dtype, tensor_id=inputs.NORM_X)
    dz = inputs.normal((rows, cols), gs, dtype, tensor_id=inputs.NORM_DZ)
    check_norm(op, dtype, x, dz, eps, f"normal({rows}x{cols})")


# One width per launch shape of the register-tile path: (waves per row, vectors per
# thread) = (1,1), (1,2), (2,2), (4,2), (4,3), (4,4), (4,6), (4,8), (4,12), (4,16), and
# the forward's (1,3) and (2,3) (its target is 3 vectors per thread, the backward's 2:
# those two widths run (2,2) and (4,2) backward).
SHAPE_WIDTHS = {"bf16": [512, 1024, 2048, 4096, 5120, 8192, 12288, 16384, 24576, 32768, 1536, 3072],
                "fp32": [256, 512, 1024, 2048, 2560, 4096, 6144, 8192, 12288, 16384, 768, 1536]}


@pytest.mark.parametrize("cols", [512, 768])
@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
@pytest.mark.parametrize("op", ["msln", "msrms"])
def test_forward_row_groups_walked_by_persistent_blocks(op, dtype, cols):
    """Rows of one wave (512 or 768 wide: one to three vectors per thread) take the
    persistent forward: with many more row groups than resident blocks, each block walks
    several groups with the next one's loads in flight and alternating LDS slots; the row
    count leaves the last group partial."""
    rows = 24003
    x = inputs.normal((rows, cols), 1.0, dtype, tensor_id=inputs.NORM_X, block=11)
    dz = inputs.normal((rows, cols), 1.0, dtype, tensor_id=inputs.NORM_DZ, block=11)
    check_norm(op, dtype, x, dz, 1e-5, f"persistent({rows}x{cols})")


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
@pytest.mark.parametrize("op", ["msln", "msrms"])
def test_every_launch_shape(op, dtype):
    for k, cols in enumerate(SHAPE_WIDTHS[dtype]):
        rows = 7  # not a multiple of the rows per block: the last block has idle rows
        x = inputs.normal((rows, cols), 1.0, dtype, tensor_id=inputs.NORM_X, block=k)
        dz = inputs.normal((rows, cols), 1.0, dtype, tensor_id=inputs.NORM_DZ, block=k)
        check_norm(op, dtype, x, dz, 1e-5, f"shape({rows}x{cols})")


@pytest.mark.parametrize("op", ["msrms", "msln"])
def test_outlier_mixture(op):
    shape = (128, 5120)
    x = inputs.outlier_mixture(shape, "bf16", tensor_id=inputs.NORM_X)
    dz = inputs.normal(shape, 1e-3, "bf16", tensor_id=inputs.NORM_DZ)
    check_norm(op, "bf16", x, dz, 1e-5, "mixture")


@pytest.mark.parametrize("shape", inputs.EDGE_SHAPES)
@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("op", ["msln", "msrms"])
def test_edge_rows(op, dtype, shape):
    """Widths 1000, 1023, 1025, 8191 with constant, zero, offset-1e4, spike and
    all-+-1e4 rows interleaved with N(0,1) rows."""
    x = inputs.edge_norm_rows(shape, dtype)
    dz = inputs.normal(shape, 1.0, dtype, tensor_id=inputs.NORM_DZ)
    check_norm(op, dtype, x, dz, inputs.EDGE_EPS[op], f"edge{shape}")


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("op", ["msln", "msrms"])
def test_misaligned_base_pointer(op, dtype):
    fwd, bwd, ofwd, obwd = NORMS[op]
    rows, cols = 33, 768
    flat = inputs.normal((rows * cols + 1,), 1.0, dtype, tensor_id=inputs.NORM_X)
    gflat = inputs.normal((rows * cols + 1,), 1.0, dtype, tensor_id=inputs.NORM_DZ)
    x = flat[1:].reshape(rows, cols)
    z_o, r_o = ofwd(oracle.decode(x, dtype), 1e-5)
    z_saved = oracle.encode(z_o, dtype)
    xt = T(flat)[1:].view(rows, cols)
    zbuf = torch.empty(rows * cols + 1, dtype=xt.dtype, device=DEV)
    z, rstd = fwd(xt, 1e-5, z=zbuf[1:].view(rows, cols))
    zflat = z_saved.reshape(-1)
    zs = T(np.concatenate([zflat[:1], zflat]))[1:].view(rows, cols)
    dzt = T(gflat)[1:].view(rows, cols)
    dx = bwd(dzt, zs, T(r_o.astype(np.float32)))
    torch.cuda.synchronize()
    rtol = rtol_for(dtype)
    assert_mixed(oracle.decode(H(z), dtype), z_o, rtol, "misaligned z")
    dx_o = obwd(oracle.decode(gflat[1:].reshape(rows, cols), dtype),
                oracle.decode(z_saved, dtype), r_o.astype(np.float32))
    assert_mixed(oracle.decode(H(dx), dtype), dx_o, rtol, "misaligned dx")


@pytest.mark.parametrize("op", ["msln", "msrms"])
def test_in_place_and_determinism(op):
    fwd, bwd, _, _ = NORMS[op]
    shape = (96, 4096)
    x = inputs.normal(shape, 1.0, "bf16", tensor_id=inputs.NORM_X)
    dz = inputs.normal(shape, 1.0, "bf16", tensor_id=inputs.NORM_DZ)
    z1, r1 = fwd(T(x), 1e-5)
    xt = T(x)
    z2, r2 = fwd(xt, 1e-5, z=xt)
    dx1 = bwd(T(dz), z1, r1)
    dzt = T(dz)
    dx2 = bwd(dzt, z1, r1, dx=dzt)
    z3, r3 = fwd(T(x), 1e-5)
    torch.cuda.synchronize()
    for a, b in ((z1, z2), (r1, r2), (z1, z3), (r1, r3), (dx1, dx2)):
        assert np.array_equal(H(a), H(b))


def test_chained_fwd_bwd_msln_fp32():
    shape = (8 * 197, 768)
    x = inputs.normal(shape, 1.0, "fp32", tensor_id=inputs.NORM_X)
    dz = inputs.normal(shape, 1.0, "fp32", tensor_id=inputs.NORM_DZ)
    z, r = lmbp.msln_fwd(T(x), 1e-6)
    dx = lmbp.msln_bwd(T(dz), z, r)
    torch.cuda.synchronize()
    z_o, r_o = oracle.msln_fwd(oracle.decode(x, "fp32"), float(np.float32(1e-6)))
    dx_o = oracle.msln_bwd(oracle.decode(dz, "fp32"), z_o, r_o)
    assert_mixed(oracle.decode(H(dx), "fp32"), dx_o, 1e-5, "chained dx")


def test_empty_rows_is_noop():
    x = torch.empty(0, 768, dtype=torch.bfloat16, device=DEV)
    z, r = lmbp.msln_fwd(x, 1e-6)
    dx = lmbp.msln_bwd(x, z, r)
    assert z.numel() == 0 and r.numel() == 0 and dx.numel() == 0
