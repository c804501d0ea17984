"""GPU parity of the table-driven k-bit family kernels (and ReGELU2-d) against the oracle."""

import numpy as np
import pytest
import torch

import oracle
from oracle import variants as OV
import paper_2406_16282_amd as lmbp
from paper_2406_16282_amd import inputs, variants
from compare import assert_codes_equal, assert_mixed, assert_rel, rtol_for

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def T(a):
    return inputs.storage_to_torch(a, DEV)


def H(t):
    return inputs.torch_to_storage(t)


def tables(bits, seed):
    r = np.random.default_rng(seed)
    m = (1 << bits) - 1
    c = np.sort(r.uniform(-5, 5, m))
    a = r.normal(0, 0.5, m - 1)
    return list(a), list(c)


def check(act, bits, a, c, dtype, x, dy, label):
    print(f"[stepact] {label}: act={act} bits={bits} dtype={dtype} shape={x.shape}", flush=True)
    rtol = rtol_for(dtype)
    lv = OV.family_levels(a)
    y_o, w_o = OV.stepact_fwd(oracle.decode(x, dtype), act, c, bits)
    dx_o = OV.stepact_bwd(oracle.decode(dy, dtype), w_o, lv, bits)
    y, codes = lmbp.stepact_fwd(T(x), act, c, bits)
    dx = lmbp.stepact_bwd(T(dy), T(w_o), variants.levels_of(a), bits)
    torch.cuda.synchronize()
    assert_codes_equal(H(codes), w_o, f"{label} codes")
    shape2 = x.shape if x.ndim == 2 else (1, x.size)
    assert_rel(oracle.decode(H(y), dtype), y_o, rtol, f"{label} y")
    assert_mixed(oracle.decode(H(y), dtype).reshape(shape2), y_o.reshape(shape2), rtol, f"{label} y mixed")
    assert_rel(oracle.decode(H(dx), dtype), dx_o, rtol, f"{label} dx", floor=0.0)


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
@pytest.mark.parametrize("bits", [1, 2, 3, 4])
@pytest.mark.parametrize("act", ["gelu", "silu"])
def test_random_tables(act, bits, dtype):
    a, c = tables(bits, seed=bits)
    for shape in ((256, 4096), (37, 1000), (1, 3)):
        x = inputs.normal(shape, 3.0, dtype, tensor_id=inputs.ACT_X)
        dy = inputs.normal(shape, 1.0, dtype, tensor_id=inputs.ACT_DY)
        check(act, bits, a, c, dtype, x, dy, f"random{shape}")


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_regelu2_d(dtype):
    shape = (512, 3072)
    x = inputs.edge_activation(shape, dtype, OV.REGELU2D_C)
    dy = inputs.normal(shape, 1.0, dtype, tensor_id=inputs.ACT_DY)
    check("gelu", 2, list(variants.REGELU2D_A), list(variants.REGELU2D_C), dtype, x, dy, "ReGELU2-d edge")


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_k2_tables_reproduce_regelu2_and_resilu2(dtype):
    """With the Appendix E tables the general kernels give the dedicated kernels' bytes."""
    shape = (300, 2048)
    for act, C, A, fwd, bwd in (("gelu", oracle.GELU_C, oracle.GELU_A, lmbp.regelu2_fwd, lmbp.regelu2_bwd),
                                ("silu", oracle.SILU_C, oracle.SILU_A, lmbp.resilu2_fwd, lmbp.resilu2_bwd)):
        x = inputs.edge_activation(shape, dtype, C)
        dy = inputs.normal(shape, 1.0, dtype, tensor_id=inputs.ACT_DY)
        y1, c1 = lmbp.stepact_fwd(T(x), act, C, 2)
        y2, c2 = fwd(T(x))
        d1 = lmbp.stepact_bwd(T(dy), c1, variants.levels_of(A), 2)
        d2 = bwd(T(dy), c2)
        torch.cuda.synchronize()
        assert np.array_equal(H(c1), H(c2))
        assert np.array_equal(H(y1), H(y2))
        assert np.array_equal(H(d1), H(d2))


def test_module_regelu2_d_autograd():
    x = torch.randn(64, 3072, device=DEV, requires_grad=True)
    y = variants.regelu2_d()(x)
    y.backward(torch.ones_like(y))
    xs = x.detach().cpu().double().numpy()
    lv = OV.family_levels(OV.REGELU2D_A)[OV.family_code(xs, OV.REGELU2D_C)]
    assert np.allclose(x.grad.cpu().double().numpy(), lv, rtol=1e-6, atol=0)


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_fitted_four_bit_gelu(dtype):
    """A k = 4 member fitted by the offline search (15 biases, 16 slopes) through the kernels."""
    from paper_2406_16282_amd import fit
    a, c, _ = fit.fit("gelu", 4, starts=1)
    shape = (128, 4096)
    x = inputs.edge_activation(shape, dtype, list(c))
    dy = inputs.normal(shape, 1.0, dtype, tensor_id=inputs.ACT_DY)
    check("gelu", 4, list(a), list(c), dtype, x, dy, "fitted k=4")


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_fitted_three_bit_silu(dtype):
    """A k = 3 member (7 biases, 8 slopes; ten codes per word) fitted by the offline search,
    on inputs crowded at its thresholds, with a ragged tail (n % 640 != 0, n % 10 = 6)."""
    from paper_2406_16282_amd import fit
    a, c, _ = fit.fit("silu", 3, starts=1)
    shape = (97, 2998)
    x = inputs.edge_activation(shape, dtype, list(c))
    dy = inputs.normal(shape, 1.0, dtype, tensor_id=inputs.ACT_DY)
    check("silu", 3, list(a), list(c), dtype, x, dy, "fitted k=3")


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_three_bit_unaligned_and_in_place(dtype):
    """k = 3 through the general path (base pointer one element off 16-byte alignment) and
    in place (y == x, dx == dy), against the oracle."""
    a, c = tables(3, seed=9)
    n = 6403
    x = inputs.normal((n + 1,), 3.0, dtype, tensor_id=inputs.ACT_X)
    dy = inputs.normal((n + 1,), 1.0, dtype, tensor_id=inputs.ACT_DY)
    lv = OV.family_levels(a)
    y_o, w_o = OV.stepact_fwd(oracle.decode(x[1:], dtype), "gelu", c, 3)
    dx_o = OV.stepact_bwd(oracle.decode(dy[1:], dtype), w_o, lv, 3)
    tx, tdy = T(x), T(dy)
    y, codes = lmbp.stepact_fwd(tx[1:], "gelu", c, 3)
    dx = lmbp.stepact_bwd(tdy[1:], T(w_o), variants.levels_of(a), 3)
    xi = T(x[1:].copy())
    lmbp.stepact_fwd(xi, "gelu", c, 3, y=xi)
    torch.cuda.synchronize()
    assert_codes_equal(H(codes), w_o, "unaligned k=3 codes")
    assert np.array_equal(H(y), H(xi)), "in-place y differs"
    rtol = rtol_for(dtype)
    assert_rel(oracle.decode(H(y), dtype), y_o, rtol, "unaligned k=3 y")
    assert_rel(oracle.decode(H(dx), dtype), dx_o, rtol, "unaligned k=3 dx", floor=0.0)
