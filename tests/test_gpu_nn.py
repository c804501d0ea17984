"""Autograd modules over the kernels, checked against the CPU oracle on the GPU."""

import numpy as np
import pytest
import torch
from torch import nn

import oracle
import paper_2406_16282_amd as lmbp
from paper_2406_16282_amd import inputs
from paper_2406_16282_amd.nn import (MSLayerNorm, MSRMSNorm, ReGELU2, ReSiLU2, ReSwiGLU2,
                                     merge_norm_into_linears)
from compare import assert_codes_equal, assert_mixed, assert_rel

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def T(a, grad=False):
    t = inputs.storage_to_torch(a, DEV)
    return t.requires_grad_(grad)


def H(t):
    return inputs.torch_to_storage(t)


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("which", ["gelu", "silu"])
def test_activation_modules(which, dtype):
    shape = (64, 3072)
    x = inputs.normal(shape, 2.0, dtype, tensor_id=inputs.ACT_X)
    dy = inputs.normal(shape, 1.0, dtype, tensor_id=inputs.ACT_DY)
    xt = T(x, True)
    y = (ReGELU2() if which == "gelu" else ReSiLU2())(xt)
    y.backward(T(dy))
    fwd = oracle.regelu2_fwd if which == "gelu" else oracle.resilu2_fwd
    bwd = oracle.regelu2_bwd if which == "gelu" else oracle.resilu2_bwd
    y_o, w_o = fwd(oracle.decode(x, dtype))
    rtol = 1e-5 if dtype == "fp32" else 1e-2
    assert_rel(oracle.decode(H(y), dtype), y_o, rtol, "module y")
    assert_rel(oracle.decode(H(xt.grad), dtype), bwd(oracle.decode(dy, dtype), w_o), rtol, "module dx", floor=0.0)


def test_swiglu_module():
    shape = (32, 11008)
    g = inputs.normal(shape, 2.0, "bf16", tensor_id=inputs.ACT_X)
    u = inputs.normal(shape, 1.0, "bf16", tensor_id=inputs.ACT_U)
    dh = inputs.normal(shape, 1.0, "bf16", tensor_id=inputs.ACT_DY)
    gt, ut = T(g, True), T(u, True)
    h = ReSwiGLU2()(gt, ut)
    h.backward(T(dh))
    h_o, s_o, w_o = oracle.reswiglu2_fwd(oracle.decode(g, "bf16"), oracle.decode(u, "bf16"))
    # The module's backward sees the s its own forward stored (bf16). That s is checked
    # against the oracle's s (one rounding); du = dh * s is then checked against the product
    # with that same stored s (one more rounding), so each rounding meets the bound once.
    _, s_gpu, _ = lmbp.reswiglu2_fwd(T(g), T(u))
    s_gpu = oracle.decode(H(s_gpu), "bf16")
    dg_o, du_o = oracle.reswiglu2_bwd(oracle.decode(dh, "bf16"), oracle.decode(u, "bf16"), s_gpu, w_o)
    assert_rel(s_gpu, s_o, 1e-2, "swiglu stored s")
    assert_rel(oracle.decode(H(h), "bf16"), h_o, 1e-2, "swiglu h")
    assert_rel(oracle.decode(H(gt.grad), "bf16"), dg_o, 1e-2, "swiglu dg")
    assert_rel(oracle.decode(H(ut.grad), "bf16"), du_o, 1e-2, "swiglu du")


@pytest.mark.parametrize("kind", ["ln", "rms"])
def test_merged_norm_linear_against_oracle(kind):
    """LayerNorm/RMSNorm with affine followed by two linear layers, merged, run through the
    MS norm kernel and torch linears in fp32; compared with the oracle norm composed with
    the same merged weights in fp64, forward and input gradient."""
    torch.manual_seed(0)
    rows, p = 96, 768
    norm = (nn.LayerNorm(p, eps=1e-6) if kind == "ln" else nn.RMSNorm(p, eps=1e-5)).to(DEV)
    with torch.no_grad():
        norm.weight.copy_(1 + 0.2 * torch.randn(p))
        if kind == "ln":
            norm.bias.copy_(0.2 * torch.randn(p))
    lins = [nn.Linear(p, 256).to(DEV), nn.Linear(p, 64).to(DEV)]
    x = inputs.normal((rows, p), 1.5, "fp32", tensor_id=inputs.NORM_X)
    dys = [inputs.normal((rows, l.out_features), 1.0, "fp32", tensor_id=10 + k) for k, l in enumerate(lins)]
    ms = merge_norm_into_linears(norm, lins)
    xt = T(x, True)
    z = ms(xt)
    ys = [l(z) for l in lins]
    sum((y * T(d)).sum() for y, d in zip(ys, dys)).backward()

    ofwd = oracle.msln_fwd if kind == "ln" else oracle.msrms_fwd
    obwd = oracle.msln_bwd if kind == "ln" else oracle.msrms_bwd
    z_o, r_o = ofwd(x.astype(np.float64), float(np.float32(ms.eps)))
    Ws = [l.weight.detach().cpu().double().numpy() for l in lins]
    bs = [l.bias.detach().cpu().double().numpy() for l in lins]
    for y, W, b in zip(ys, Ws, bs):
        assert_mixed(H(y).astype(np.float64), z_o @ W.T + b, 1e-5, f"{kind} merged y")
    dz_o = sum(d.astype(np.float64) @ W for d, W in zip(dys, Ws))
    assert_mixed(H(xt.grad).astype(np.float64), obwd(dz_o, z_o, r_o), 1e-5, f"{kind} merged dx")


def test_norm_saves_only_z_shared_with_the_linear_and_rstd():
    """Memory sharing (Prop. 5.1): the tensors autograd saves for MS-LN followed by a
    linear layer are z (saved once, by both), rstd and the weight."""
    p = 512
    ms, lin = MSLayerNorm(1e-6), nn.Linear(p, 128).to(DEV)
    x = torch.randn(64, p, device=DEV, requires_grad=True)
    saved = []
    with torch.autograd.graph.saved_tensors_hooks(lambda t: (saved.append(t), t)[1], lambda t: t):
        z = ms(x)
        y = lin(z)
    ptrs = {t.data_ptr(): t for t in saved}
    act = [t for t in ptrs.values() if t.data_ptr() != lin.weight.data_ptr()]
    assert sorted(tuple(t.shape) for t in act) == [(64,), (64, p)]
    assert any(t.data_ptr() == z.data_ptr() for t in act)


def test_activation_saves_only_codes():
    x = torch.randn(256, 1024, device=DEV, dtype=torch.bfloat16, requires_grad=True)
    saved = []
    with torch.autograd.graph.saved_tensors_hooks(lambda t: (saved.append(t), t)[1], lambda t: t):
        ReSiLU2()(x)
    assert len(saved) == 1 and saved[0].dtype == torch.int32
    assert saved[0].numel() * 4 == x.numel() // 4   # 2 bits per element


@pytest.mark.parametrize("which", ["gelu", "silu"])
def test_fused_linear_act_module(which):
    """LinearReGELU2 / LinearReSiLU2 against the oracle: forward (stored z rounding, y),
    and the Approx-BP gradients dx = (dy * slope[code(z)]) W, dW = (dy * slope)^T x,
    db = sum(dy * slope), computed in fp64 from the oracle's codes of the rounded z.
    Dyadic inputs make the GPU's fp32 accumulation of z exact, so the codes agree."""
    from paper_2406_16282_amd.nn import LinearReGELU2, LinearReSiLU2
    m, k, n = 96, 64, 160
    x = inputs.dyadic((m, k), -3, tensor_id=inputs.LIN_X)
    w = inputs.dyadic((n, k), -4, tensor_id=inputs.LIN_W)
    b = inputs.dyadic((n,), -7, tensor_id=inputs.LIN_B)
    dy = inputs.normal((m, n), 1.0, "bf16", tensor_id=inputs.ACT_DY)
    mod = (LinearReGELU2 if which == "gelu" else LinearReSiLU2)(k, n, device=DEV)
    with torch.no_grad():
        mod.weight.copy_(T(w))
        mod.bias.copy_(T(b))
    xt = T(x, True)
    y = mod(xt)
    y.backward(T(dy))
    _, z_s, y_o, c_o = oracle.linear_act_fwd(x, w, b, which)
    assert_rel(oracle.decode(H(y), "bf16"), y_o, 1e-2, "fused module y")
    obwd = oracle.regelu2_bwd if which == "gelu" else oracle.resilu2_bwd
    dz = oracle.decode(oracle.encode(obwd(oracle.decode(dy, "bf16"), c_o), "bf16"), "bf16")
    xd, wd = oracle.decode(x, "bf16"), oracle.decode(w, "bf16")
    assert_mixed(oracle.decode(H(xt.grad), "bf16"), dz @ wd, 1e-2, "fused module dx")
    assert_mixed(oracle.decode(H(mod.weight.grad), "bf16"), dz.T @ xd, 1e-2, "fused module dW")
    assert_mixed(oracle.decode(H(mod.bias.grad), "bf16").reshape(1, -1), dz.sum(0).reshape(1, -1),
                 1e-2, "fused module db")



def test_fused_linear_swiglu_module():
    """LinearReSwiGLU2 against the oracle: forward h, and the Approx-BP gradients
    dg = dh * u * slope[code(g)], du = dh * s, dx = dg Wg + du Wu, dWg = dg^T x, dWu = du^T x
    (fp64 from the oracle's stored g, u). Dyadic inputs keep the GPU's g and u exact."""
    from paper_2406_16282_amd.nn import LinearReSwiGLU2
    m, k, n = 96, 64, 80
    x = inputs.dyadic((m, k), -3, tensor_id=inputs.LIN_X)
    wg = inputs.dyadic((n, k), -4, tensor_id=inputs.LIN_W)
    wu = inputs.dyadic((n, k), -4, tensor_id=inputs.LIN_B)
    dh = inputs.normal((m, n), 1.0, "bf16", tensor_id=inputs.ACT_DY)
    mod = LinearReSwiGLU2(k, n, device=DEV)
    with torch.no_grad():
        mod.gate.weight.copy_(T(wg))
        mod.up.weight.copy_(T(wu))
    xt = T(x, True)
    h = mod(xt)
    h.backward(T(dh))
    _, g_s, _, u_s, h_o, s_o, c_o = oracle.linear_swiglu_fwd(x, wg, wu)
    assert_mixed(oracle.decode(H(h), "bf16"), h_o, 1e-2, "swiglu module h")
    s_st = oracle.decode(oracle.encode(s_o, "bf16"), "bf16")
    dg_o, du_o = oracle.reswiglu2_bwd(oracle.decode(dh, "bf16"), oracle.decode(u_s, "bf16"), s_st, c_o)
    dg_o = oracle.decode(oracle.encode(dg_o, "bf16"), "bf16")
    du_o = oracle.decode(oracle.encode(du_o, "bf16"), "bf16")
    xd, wgd, wud = (oracle.decode(a, "bf16") for a in (x, wg, wu))
    assert_mixed(oracle.decode(H(xt.grad), "bf16"), dg_o @ wgd + du_o @ wud, 1e-2, "swiglu module dx")
    assert_mixed(oracle.decode(H(mod.gate.weight.grad), "bf16"), dg_o.T @ xd, 1e-2, "swiglu module dWg")
    assert_mixed(oracle.decode(H(mod.up.weight.grad), "bf16"), du_o.T @ xd, 1e-2, "swiglu module dWu")


def _saved_activation_bytes(run, params):
    """Bytes of the distinct tensors autograd saves during `run()`, parameters excluded
    (tensors sharing storage are counted once, as autograd keeps them once)."""
    saved = []
    with torch.autograd.graph.saved_tensors_hooks(lambda t: (saved.append(t), t)[1], lambda t: t):
        out = run()
    skip = {p.data_ptr() for p in params}
    storages = {}
    for t in saved:
        st = t.untyped_storage()
        if t.data_ptr() in skip:
            continue
        storages[st.data_ptr()] = st.nbytes()
    return sum(storages.values()), out


def test_vit_mlp_block_activation_memory():
    """A ViT-B MLP block (norm, 768 -> 3072, GELU, 3072 -> 768; bf16, 256 tokens): the
    standard torch block against MS-LN + ReGELU2 (Sec. 4-5), unfused and with the fused
    linear + activation. Ours keeps, per token, z (2p B, shared by the norm and fc1), rstd
    (4 B), the 2-bit codes (F/4 B) and fc2's input (2F B), exactly."""
    from paper_2406_16282_amd.nn import LinearReGELU2
    tok, p, f = 256, 768, 3072
    x = torch.randn(tok, p, device=DEV, dtype=torch.bfloat16)
    ln = nn.LayerNorm(p, eps=1e-6, device=DEV, dtype=torch.bfloat16)
    fc1 = nn.Linear(p, f, device=DEV, dtype=torch.bfloat16)
    fc2 = nn.Linear(f, p, device=DEV, dtype=torch.bfloat16)
    xs = x.clone().requires_grad_(True)
    std, _ = _saved_activation_bytes(lambda: fc2(nn.functional.gelu(fc1(ln(xs)))),
                                     list(ln.parameters()) + list(fc1.parameters()) + list(fc2.parameters()))
    ms = MSLayerNorm(1e-6)
    act = ReGELU2()
    params = list(fc1.parameters()) + list(fc2.parameters())
    xo = x.clone().requires_grad_(True)
    ours, _ = _saved_activation_bytes(lambda: fc2(act(fc1(ms(xo)))), params)
    fused = LinearReGELU2(p, f, device=DEV)
    xf = x.clone().requires_grad_(True)
    ours_fused, _ = _saved_activation_bytes(lambda: fc2(fused(ms(xf))),
                                            params + list(fused.parameters()))
    want = tok * (2 * p + 4 + f // 4 + 2 * f)
    print(f"[nn] ViT-B MLP block saved bytes per token: torch {std / tok:.0f}, "
          f"MS-LN + ReGELU2 {ours / tok:.0f}, fused {ours_fused / tok:.0f}", flush=True)
    assert ours == want and ours_fused == want
    assert std >= tok * (4 * p + 4 * f)       # x, norm output, fc1 output, GELU output
    assert ours / std < 0.56


def test_llama_mlp_block_activation_memory():
    """A LLaMA-7B MLP block (RMSNorm, gate and up 4096 -> 11008, SwiGLU, down 11008 -> 4096;
    bf16, 64 tokens): standard torch against MS-RMSNorm + ReSwiGLU2 (unfused) and the fused
    gate/up + SwiGLU layer. Ours keeps z (2p, shared), rstd (4), codes of g (F/4), u and
    s = SiLU(g) (2F each), and the down projection's input h (2F) per token."""
    from paper_2406_16282_amd.nn import LinearReSwiGLU2
    tok, p, f = 64, 4096, 11008
    x = torch.randn(tok, p, device=DEV, dtype=torch.bfloat16)
    rms = nn.RMSNorm(p, eps=1e-5, device=DEV, dtype=torch.bfloat16)
    gate = nn.Linear(p, f, bias=False, device=DEV, dtype=torch.bfloat16)
    up = nn.Linear(p, f, bias=False, device=DEV, dtype=torch.bfloat16)
    down = nn.Linear(f, p, bias=False, device=DEV, dtype=torch.bfloat16)
    params = [gate.weight, up.weight, down.weight]
    xs = x.clone().requires_grad_(True)

    def standard():
        z = rms(xs)
        return down(nn.functional.silu(gate(z)) * up(z))
    std, _ = _saved_activation_bytes(standard, params + [rms.weight])
    ms, glu = MSRMSNorm(1e-5), ReSwiGLU2()
    xo = x.clone().requires_grad_(True)

    def ours_fn():
        z = ms(xo)
        return down(glu(gate(z), up(z)))
    ours, _ = _saved_activation_bytes(ours_fn, params)
    fused = LinearReSwiGLU2(p, f, device=DEV)
    xf = x.clone().requires_grad_(True)
    ours_fused, _ = _saved_activation_bytes(lambda: down(fused(ms(xf))),
                                            params + [fused.gate.weight, fused.up.weight])
    print(f"[nn] LLaMA-7B MLP block saved bytes per token: torch {std / tok:.0f}, "
          f"MS-RMSNorm + ReSwiGLU2 {ours / tok:.0f}, fused {ours_fused / tok:.0f}", flush=True)
    assert ours_fused == tok * (2 * p + 4 + f // 4 + 3 * 2 * f)
    assert ours == ours_fused
    assert ours < std
