"""Other members of the ReLU-combination family for the table-driven kernels.

A member is given by weights a_1..a_{m-1} (the last weight is 1 - sum a) and
increasing biases c_1..c_m, m = 2^k - 1 (eq. relus_family). Its step derivative has
2^k levels, the cumulative sums of the weights (Prop. 4.3); ``stepact_fwd`` takes the
biases as thresholds and ``stepact_bwd`` the levels.
"""

import torch
from torch import nn

from . import binding

# Appendix I: ReGELU2-d, the k = 2 member fitted to GELU's derivative.
REGELU2D_A = (0.32465931184406527, 0.34812875668739607)
REGELU2D_C = (-0.4535743722857079, -0.0010587205574873046, 0.4487575313884231)


def levels_of(a):
    """The 2^k slopes of the combination with weights a (last slope exactly 1)."""
    out, acc = [0.0], 0.0
    for w in a:
        acc += float(w)
        out.append(acc)
    out.append(1.0)
    return out


def bits_of(c):
    m = len(c)
    for k in (1, 2, 3, 4):
        if m == (1 << k) - 1:
            return k
    raise ValueError("the number of biases must be 1, 3, 7 or 15 (k = 1, 2, 3, 4)")


class _Step(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x, act, c, levels, bits):
        y, codes = binding.stepact_fwd(x.contiguous(), act, c, bits)
        ctx.levels, ctx.bits = levels, bits
        ctx.save_for_backward(codes)
        return y

    @staticmethod
    def backward(ctx, dy):
        (codes,) = ctx.saved_tensors
        return binding.stepact_bwd(dy.contiguous(), codes, ctx.levels, ctx.bits), None, None, None, None


class StepActivation(nn.Module):
    """Exact GELU/SiLU forward; backward through the step derivative of the family
    member (a, c), saving k bits per element."""

    def __init__(self, act, a, c):
        super().__init__()
        if act not in ("gelu", "silu"):
            raise ValueError("act must be 'gelu' or 'silu'")
        if len(a) + 1 != len(c):
            raise ValueError("need len(a) + 1 == len(c)")
        self.act, self.c = act, tuple(float(v) for v in c)
        self.bits = bits_of(self.c)
        self.levels = tuple(levels_of(a))

    def forward(self, x):
        return _Step.apply(x, self.act, self.c, self.levels, self.bits)

    def extra_repr(self):
        return f"act={self.act}, bits={self.bits}"


def regelu2_d():
    """ReGELU2-d of Appendix I."""
    return StepActivation("gelu", REGELU2D_A, REGELU2D_C)
