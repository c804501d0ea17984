"""The affine merge of Sec. 5.2 on the CPU (torch float64 reference norms; no kernels):
norm with affine (alpha, beta) followed by Linear(W, b) equals the parameter-free norm
followed by the merged Linear(W diag(alpha), W beta + b)."""

import copy

import pytest
import torch
import torch.nn.functional as F
from torch import nn

from paper_2406_16282_amd.nn import MSLayerNorm, MSRMSNorm, merge_norm_into_linears


def _setup(kind, p=48, q=(20, 7), seed=0):
    g = torch.Generator().manual_seed(seed)
    norm = nn.LayerNorm(p, eps=1e-6, dtype=torch.float64) if kind == "ln" else nn.RMSNorm(p, eps=1e-5, dtype=torch.float64)
    with torch.no_grad():
        norm.weight.copy_(1 + 0.3 * torch.randn(p, generator=g, dtype=torch.float64))
        if kind == "ln":
            norm.bias.copy_(0.3 * torch.randn(p, generator=g, dtype=torch.float64))
    lins = [nn.Linear(p, k, dtype=torch.float64) for k in q]
    x = torch.randn(9, p, generator=g, dtype=torch.float64) * 1.7 + 0.2
    return norm, lins, x


@pytest.mark.parametrize("kind", ["ln", "rms"])
def test_merged_layers_compute_the_same_function(kind):
    norm, lins, x = _setup(kind)
    ref = [lin(norm(x)) for lin in lins]
    merged = [copy.deepcopy(l) for l in lins]
    ms = merge_norm_into_linears(copy.deepcopy(norm), merged)
    assert isinstance(ms, MSLayerNorm if kind == "ln" else MSRMSNorm)
    assert ms.eps == norm.eps
    z = F.layer_norm(x, (x.shape[1],), eps=ms.eps) if kind == "ln" else F.rms_norm(x, (x.shape[1],), eps=ms.eps)
    for r, lin in zip(ref, merged):
        assert torch.allclose(lin(z), r, rtol=0, atol=1e-12)


def test_merge_creates_bias_when_missing():
    norm, _, x = _setup("ln")
    lin = nn.Linear(48, 5, bias=False, dtype=torch.float64)
    ref = lin(norm(x))
    merged = copy.deepcopy(lin)
    merge_norm_into_linears(norm, [merged])
    assert merged.bias is not None
    z = F.layer_norm(x, (48,), eps=1e-6)
    assert torch.allclose(merged(z), ref, atol=1e-12)


def test_merge_rejects_multi_dim_norms():
    with pytest.raises(ValueError):
        merge_norm_into_linears(nn.LayerNorm((4, 8)), [nn.Linear(8, 2)])
    with pytest.raises(TypeError):
        merge_norm_into_linears(nn.BatchNorm1d(8), [nn.Linear(8, 2)])
