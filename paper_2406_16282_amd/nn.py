"""Autograd modules over the lmbp kernels, and the affine merge that enables MS-BP.

* ``ReGELU2`` / ``ReSiLU2``: exact GELU / SiLU forward, 2-bit codes saved, step
  derivative backward (Sec. 4.2).
* ``ReSwiGLU2``: h = SiLU(g) * u with ReSiLU2's backward for the SiLU factor (the LLaMA
  MLP, Sec. 6); saves the codes and s = SiLU(g).
* ``MSLayerNorm`` / ``MSRMSNorm``: parameter-free norms (Sec. 5.2, Appendix G) that save
  only their output z and one fp32 rstd per row. z is the same tensor the following
  linear layer saves as its input, so autograd keeps one copy (memory sharing).
* ``LinearReGELU2`` / ``LinearReSiLU2``: a bf16 linear layer followed by the activation,
  forward fused into one kernel (the pre-activation is never stored); saves x (for the
  weight gradient) and the codes. Backward: dz = dy * slope[code] by the activation
  kernel, then the two products of a linear layer's backward (library GEMMs).
* ``LinearReSwiGLU2``: the LLaMA MLP's gate and up projections with SwiGLU, forward fused
  in one kernel (g never stored); backward through the SwiGLU activation backward and
  the linear layers' products.
* ``merge_norm_into_linears``: folds a norm's affine (alpha, beta) into the linear layers
  that consume its output, W~ = W diag(alpha), b~ = W beta + b (Sec. 5.2), and returns
  the parameter-free MS norm to use in its place.

Every forward and backward runs in the HIP kernels through ``binding``, except the two
matrix products of the fused linear layer's backward (torch's library GEMMs) and the
one-time weight merge.
"""

import torch
from torch import nn

from . import binding


def _flat(t):
    return t if t.is_contiguous() else t.contiguous()


class _Act(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x, which):
        fwd = binding.regelu2_fwd if which == "gelu" else binding.resilu2_fwd
        y, codes = fwd(_flat(x))
        ctx.which = which
        ctx.save_for_backward(codes)
        return y

    @staticmethod
    def backward(ctx, dy):
        (codes,) = ctx.saved_tensors
        bwd = binding.regelu2_bwd if ctx.which == "gelu" else binding.resilu2_bwd
        return bwd(_flat(dy), codes), None


class _SwiGLU(torch.autograd.Function):
    @staticmethod
    def forward(ctx, g, u):
        g, u = _flat(g), _flat(u)
        if g.shape != u.shape:
            raise ValueError("g and u must have the same shape")
        h, s, codes = binding.reswiglu2_fwd(g, u)
        ctx.save_for_backward(u, s, codes)
        return h

    @staticmethod
    def backward(ctx, dh):
        u, s, codes = ctx.saved_tensors
        dg, du = binding.reswiglu2_bwd(_flat(dh), u, s, codes)
        return dg, du


class _MSNorm(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x, eps, centered):
        fwd = binding.msln_fwd if centered else binding.msrms_fwd
        z, rstd = fwd(_flat(x), eps)
        ctx.centered = centered
        ctx.save_for_backward(z, rstd)
        return z

    @staticmethod
    def backward(ctx, dz):
        z, rstd = ctx.saved_tensors
        bwd = binding.msln_bwd if ctx.centered else binding.msrms_bwd
        return bwd(_flat(dz), z, rstd), None, None


class _LinearAct(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x, weight, bias, which):
        x2 = _flat(x).reshape(-1, x.shape[-1])
        y, codes = binding.linear_act_fwd(x2, _flat(weight), None if bias is None else _flat(bias),
                                          act=which)
        ctx.which = which
        ctx.has_bias = bias is not None
        ctx.x_shape = x.shape
        ctx.save_for_backward(x2, weight, codes)
        return y.reshape(*x.shape[:-1], weight.shape[0])

    @staticmethod
    def backward(ctx, dy):
        x2, weight, codes = ctx.saved_tensors
        bwd = binding.regelu2_bwd if ctx.which == "gelu" else binding.resilu2_bwd
        dz = bwd(_flat(dy).reshape(-1, weight.shape[0]), codes)
        # The two products of a linear layer's backward, as torch's own linear layer forms
        # them (2-D GEMMs; the transposed left operand is read in place by the library).
        dx = (dz @ weight).reshape(ctx.x_shape) if ctx.needs_input_grad[0] else None
        dw = dz.t().mm(x2) if ctx.needs_input_grad[1] else None
        db = dz.sum(0, dtype=torch.float32).to(dz.dtype) if ctx.has_bias and ctx.needs_input_grad[2] else None
        return dx, dw, db, None


class _LinearActModule(nn.Linear):
    """bf16 nn.Linear whose output goes through the activation, fused. Output features
    must be a multiple of 16, input features a multiple of 8."""
    which = None

    def __init__(self, in_features, out_features, bias=True, device=None, dtype=torch.bfloat16):
        super().__init__(in_features, out_features, bias=bias, device=device, dtype=dtype)

    def forward(self, x):
        return _LinearAct.apply(x, self.weight, self.bias, self.which)


class LinearReGELU2(_LinearActModule):
    """GELU(x W^T + b) with ReGELU2's backward (Sec. 4.2), forward fused in one kernel."""
    which = "gelu"


class LinearReSiLU2(_LinearActModule):
    """SiLU(x W^T + b) with ReSiLU2's backward (Sec. 4.2), forward fused in one kernel."""
    which = "silu"


class _LinearSwiGLU(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x, w_gate, w_up):
        x2 = _flat(x).reshape(-1, x.shape[-1])
        h, s, u, codes = binding.linear_swiglu_fwd(x2, _flat(w_gate), _flat(w_up))
        ctx.x_shape = x.shape
        ctx.save_for_backward(x2, w_gate, w_up, s, u, codes)
        return h.reshape(*x.shape[:-1], w_gate.shape[0])

    @staticmethod
    def backward(ctx, dh):
        x2, w_gate, w_up, s, u, codes = ctx.saved_tensors
        dg, du = binding.reswiglu2_bwd(_flat(dh).reshape(-1, w_gate.shape[0]), u, s, codes)
        dx = torch.addmm(dg @ w_gate, du, w_up).reshape(ctx.x_shape) if ctx.needs_input_grad[0] else None
        dwg = dg.t().mm(x2) if ctx.needs_input_grad[1] else None
        dwu = du.t().mm(x2) if ctx.needs_input_grad[2] else None
        return dx, dwg, dwu


class LinearReSwiGLU2(nn.Module):
    """The LLaMA MLP's input side, SiLU(x Wg^T) * (x Wu^T), with ReSiLU2's backward for
    the SiLU factor; forward fused in one kernel (bf16; out_features a multiple of 16,
    in_features of 8). Saves x, s = SiLU(g), u and the codes of g."""

    def __init__(self, in_features, out_features, device=None, dtype=torch.bfloat16):
        super().__init__()
        self.gate = nn.Linear(in_features, out_features, bias=False, device=device, dtype=dtype)
        self.up = nn.Linear(in_features, out_features, bias=False, device=device, dtype=dtype)

    def forward(self, x):
        return _LinearSwiGLU.apply(x, self.gate.weight, self.up.weight)


class ReGELU2(nn.Module):
    """GELU forward; backward through the 2-bit step derivative (Sec. 4.2)."""

    def forward(self, x):
        return _Act.apply(x, "gelu")


class ReSiLU2(nn.Module):
    """SiLU forward; backward through the 2-bit step derivative (Sec. 4.2)."""

    def forward(self, x):
        return _Act.apply(x, "silu")


class ReSwiGLU2(nn.Module):
    """h = SiLU(g) * u with ReSiLU2's backward for the SiLU factor."""

    def forward(self, g, u):
        return _SwiGLU.apply(g, u)


class MSLayerNorm(nn.Module):
    """LayerNorm without affine over the last dimension, saving only z and rstd
    (Alg. 1 / Alg. 2). Use after merging the affine into the next linear layers."""

    def __init__(self, eps=1e-6):
        super().__init__()
        self.eps = float(eps)

    def forward(self, x):
        return _MSNorm.apply(x, self.eps, True)

    def extra_repr(self):
        return f"eps={self.eps}"


class MSRMSNorm(nn.Module):
    """RMSNorm without weight over the last dimension, saving only z and rstd (Alg. 3)."""

    def __init__(self, eps=1e-5):
        super().__init__()
        self.eps = float(eps)

    def forward(self, x):
        return _MSNorm.apply(x, self.eps, False)

    def extra_repr(self):
        return f"eps={self.eps}"


@torch.no_grad()
def merge_affine_into_linear(linear, alpha, beta=None):
    """In place: W <- W diag(alpha); b <- W beta + b (Sec. 5.2). The products are formed
    in float64 and rounded once to the layer's dtype. A bias is created if beta is
    given and the layer had none."""
    W = linear.weight
    if W.shape[1] != alpha.numel():
        raise ValueError("alpha must have one entry per input feature of the linear layer")
    W64 = W.double()
    a64 = alpha.detach().to(W.device, torch.float64).reshape(-1)
    if beta is not None:
        b_add = W64 @ beta.detach().to(W.device, torch.float64).reshape(-1)
        if linear.bias is None:
            linear.bias = nn.Parameter(b_add.to(W.dtype))
        else:
            linear.bias.copy_((linear.bias.double() + b_add).to(linear.bias.dtype))
    W.copy_((W64 * a64[None, :]).to(W.dtype))
    return linear


@torch.no_grad()
def merge_norm_into_linears(norm, linears):
    """Fold the affine of ``norm`` (a torch LayerNorm or RMSNorm with elementwise
    affine) into every linear layer that consumes its output, and return the
    parameter-free MS norm that replaces it. Requires normalization over one
    (the last) dimension."""
    if not isinstance(norm, (nn.LayerNorm, nn.RMSNorm)):
        raise TypeError("norm must be torch.nn.LayerNorm or torch.nn.RMSNorm")
    shape = tuple(norm.normalized_shape)
    if len(shape) != 1:
        raise ValueError("only normalization over the last dimension is supported")
    alpha = norm.weight if norm.weight is not None else torch.ones(shape[0])
    if isinstance(norm, nn.LayerNorm):
        beta = norm.bias
        ms = MSLayerNorm(norm.eps)
    elif isinstance(norm, nn.RMSNorm):
        beta = None
        eps = norm.eps if norm.eps is not None else torch.finfo(torch.float32).eps
        ms = MSRMSNorm(eps)
    for lin in linears:
        merge_affine_into_linear(lin, alpha, beta)
    return ms
