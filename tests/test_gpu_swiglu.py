"""GPU parity of ReSiLU2 fused with the SwiGLU product against the CPU oracle."""

import numpy as np
import pytest
import torch

import oracle
import paper_2406_16282_amd as lmbp
from paper_2406_16282_amd import inputs
from compare import NORMAL_MIN, assert_codes_equal, assert_mixed, assert_rel, rtol_for

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def T(a):
    return inputs.storage_to_torch(a, DEV)


def H(t):
    return inputs.torch_to_storage(t)


def check(dtype, g, u, dh, label):
    print(f"[swiglu] {label}: dtype={dtype} shape={g.shape}", flush=True)
    rtol = rtol_for(dtype)
    h_o, s_o, w_o = oracle.reswiglu2_fwd(oracle.decode(g, dtype), oracle.decode(u, dtype))
    s_saved = oracle.encode(s_o, dtype)
    dg_o, du_o = oracle.reswiglu2_bwd(oracle.decode(dh, dtype), oracle.decode(u, dtype),
                                      oracle.decode(s_saved, dtype), w_o)
    h, s, codes = lmbp.reswiglu2_fwd(T(g), T(u))
    dg, du = lmbp.reswiglu2_bwd(T(dh), T(u), T(s_saved), T(w_o))
    torch.cuda.synchronize()
    shape2 = g.shape if g.ndim == 2 else (1, g.size)
    assert_codes_equal(H(codes), w_o, f"{label} codes")
    dec = lambda t: oracle.decode(H(t), dtype).reshape(shape2)
    assert_rel(dec(s), s_o.reshape(shape2), rtol, f"{label} s (strict)")
    assert_mixed(dec(h), h_o.reshape(shape2), rtol, f"{label} h")
    assert_rel(dec(h), h_o.reshape(shape2), rtol, f"{label} h (strict)")
    assert_mixed(dec(dg), dg_o.reshape(shape2), rtol, f"{label} dg")
    # products of two storage values can fall below the smallest normal (and below bf16's
    # subnormal range): those are held to the mixed rule only, as forward outputs are
    assert_rel(dec(dg), dg_o.reshape(shape2), rtol, f"{label} dg (strict)")
    assert_mixed(dec(du), du_o.reshape(shape2), rtol, f"{label} du")
    zero = oracle.unpack_codes(w_o, g.size).reshape(shape2) == 0
    assert np.all(dec(dg)[zero] == 0.0), "code-0 gradients must be exactly zero"


CASES = [("bf16", (512, 11008)), ("fp32", (300, 11008)), ("bf16", (37, 1000)),
         ("fp32", (1, 17)), ("bf16", (3, 2049)), ("bf16", (1, 1))]


@pytest.mark.parametrize("dtype,shape", CASES)
def test_parity(dtype, shape):
    g = inputs.normal(shape, 2.0, dtype, tensor_id=inputs.ACT_X)
    u = inputs.normal(shape, 1.0, dtype, tensor_id=inputs.ACT_U)
    dh = inputs.normal(shape, 1e-3, dtype, tensor_id=inputs.ACT_DY)
    check(dtype, g, u, dh, f"normal{shape}")


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("shape", inputs.EDGE_SHAPES[:2])
def test_edge_gate_values(dtype, shape):
    g = inputs.edge_activation(shape, dtype, oracle.SILU_C)
    u = inputs.normal(shape, 1.0, dtype, tensor_id=inputs.ACT_U)
    dh = inputs.normal(shape, 1.0, dtype, tensor_id=inputs.ACT_DY)
    check(dtype, g, u, dh, f"edge{shape}")


def test_in_place_and_misaligned():
    n = 3 * 4096 + 5
    g = inputs.normal((n + 1,), 2.0, "bf16", tensor_id=inputs.ACT_X)
    u = inputs.normal((n + 1,), 1.0, "bf16", tensor_id=inputs.ACT_U)
    dh = inputs.normal((n + 1,), 1.0, "bf16", tensor_id=inputs.ACT_DY)
    # reference results from separate buffers
    h1, s1, c1 = lmbp.reswiglu2_fwd(T(g), T(u))
    dg1, du1 = lmbp.reswiglu2_bwd(T(dh), T(u), s1, c1)
    # in place: h over g, dg over dh, du over u
    gt, ut, dht = T(g), T(u), T(dh)
    h2, s2, c2 = lmbp.reswiglu2_fwd(gt, ut, h=gt)
    dg2, du2 = lmbp.reswiglu2_bwd(dht, ut, s2, c2, dg=dht, du=ut)
    # misaligned views (one element past a 16-byte boundary): general path
    gm, um, dhm = T(g)[1:], T(u)[1:], T(dh)[1:]
    h3, s3, c3 = lmbp.reswiglu2_fwd(gm, um)
    torch.cuda.synchronize()
    for a, b in ((h1, h2), (s1, s2), (c1, c2), (dg1, dg2), (du1, du2)):
        assert np.array_equal(H(a), H(b))
    h_o, s_o, w_o = oracle.reswiglu2_fwd(oracle.decode(g[1:], "bf16"), oracle.decode(u[1:], "bf16"))
    assert_codes_equal(H(c3), w_o, "misaligned codes")
    assert_rel(oracle.decode(H(h3), "bf16"), h_o, 1e-2, "misaligned h")


@pytest.mark.parametrize("name", ["llama7b_swiglu_bf16", "llama13b_outliers_bf16"])
def test_full_size(name):
    """Every element of h, s, codes, dg and du at the full LLaMA gate sizes, compared on
    the host in blocks of rows. The backward is fed the oracle's saved state (s rounded
    to the storage format, codes)."""
    w = inputs.WORKLOADS[name]
    sp = w.act
    print(f"[swiglu full] {name}: [{sp.rows}x{sp.cols}]", flush=True)
    g = w.act_x().reshape(sp.rows, sp.cols)
    u = w.act_u().reshape(sp.rows, sp.cols)
    dh = w.act_dy().reshape(sp.rows, sp.cols)
    h, sv, codes = lmbp.reswiglu2_fwd(T(g), T(u))
    torch.cuda.synchronize()
    h_h, s_h, c_h = H(h).reshape(sp.rows, sp.cols), H(sv).reshape(sp.rows, sp.cols), H(codes)
    del h, sv, codes
    step = max(1, (8 << 20) // sp.cols)
    per_row = sp.cols // 16
    s_saved = np.empty_like(g)
    w_all = []
    rtol = rtol_for(sp.dtype)
    for r0 in range(0, sp.rows, step):
        r1 = min(sp.rows, r0 + step)
        u64 = oracle.decode(u[r0:r1], sp.dtype)
        h_o, s_o, w_o = oracle.reswiglu2_fwd(oracle.decode(g[r0:r1], sp.dtype), u64)
        assert_codes_equal(c_h[r0 * per_row:r1 * per_row], w_o, f"{name} codes rows {r0}:{r1}")
        assert_rel(oracle.decode(s_h[r0:r1], sp.dtype), s_o, rtol, f"{name} s rows {r0}:{r1}")
        assert_rel(oracle.decode(h_h[r0:r1], sp.dtype), h_o, rtol, f"{name} h rows {r0}:{r1}")
        s_saved[r0:r1] = oracle.encode(s_o, sp.dtype)
        w_all.append(w_o)
    del h_h, s_h
    w_all = np.concatenate(w_all)
    dg, du = lmbp.reswiglu2_bwd(T(dh), T(u), T(s_saved), T(w_all))
    torch.cuda.synchronize()
    dg_h, du_h = H(dg).reshape(sp.rows, sp.cols), H(du).reshape(sp.rows, sp.cols)
    for r0 in range(0, sp.rows, step):
        r1 = min(sp.rows, r0 + step)
        dg_o, du_o = oracle.reswiglu2_bwd(oracle.decode(dh[r0:r1], sp.dtype), oracle.decode(u[r0:r1], sp.dtype),
                                          oracle.decode(s_saved[r0:r1], sp.dtype),
                                          w_all[r0 * per_row:r1 * per_row])
        assert_rel(oracle.decode(dg_h[r0:r1], sp.dtype), dg_o, rtol, f"{name} dg rows {r0}:{r1}")
        assert_rel(oracle.decode(du_h[r0:r1], sp.dtype), du_o, rtol, f"{name} du rows {r0}:{r1}")
        assert np.all(oracle.decode(dg_h[r0:r1], sp.dtype)[dg_o == 0] == 0), "code-0 gradients must be zero"
    print(f"[swiglu full] {name}: all {sp.rows * sp.cols} elements compared", flush=True)
