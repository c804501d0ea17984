"""The hot-path kernels under HIP graph capture: the library enqueues plain kernel
launches on the caller's stream (no allocation, no memset, no synchronisation), so a
captured sequence replays to the same bytes as eager launches. Each replay is checked
against the eager result, with eager work and synchronisations between replays."""

import numpy as np
import pytest
import torch

import paper_2406_16282_amd as lmbp
from paper_2406_16282_amd import inputs

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def T(a):
    return inputs.storage_to_torch(a, DEV)


# k-bit family tables for k = 3 and 4 (evenly spaced biases; any increasing table will do).
_C3 = [-2.0 + i * (4.0 / 6) for i in range(7)]
_L3 = [i / 7 for i in range(8)]
_C4 = [-3.0 + i * (6.0 / 14) for i in range(15)]
_L4 = [i / 15 for i in range(16)]


def _step(t, out):
    """MS-RMSNorm and MS-LN fwd / bwd, ReSiLU2 fwd / bwd, the fused SwiGLU pair, the
    k = 3 and k = 4 family kernels and (bf16) the fused linear layer, writing into the
    preallocated ``out`` tensors on the current stream."""
    lmbp.msrms_fwd(t["x"], 1e-5, z=out["z"], rstd=out["rstd"])
    lmbp.resilu2_fwd(t["g"], y=out["y"], codes=out["codes"])
    lmbp.resilu2_bwd(t["dy"], out["codes"], dx=out["dg"])
    lmbp.msrms_bwd(t["dz"], out["z"], out["rstd"], dx=out["dx"])
    lmbp.reswiglu2_fwd(t["g"], t["u"], h=out["h"], s=out["s"], codes=out["codes2"])
    lmbp.reswiglu2_bwd(t["dy"], t["u"], out["s"], out["codes2"], dg=out["dg2"], du=out["du2"])
    lmbp.msln_fwd(t["x"], 1e-6, z=out["zl"], rstd=out["rstdl"])
    lmbp.msln_bwd(t["dz"], out["zl"], out["rstdl"], dx=out["dxl"])
    lmbp.stepact_fwd(t["g"], "gelu", _C3, 3, y=out["y3"], codes=out["codes3"])
    lmbp.stepact_bwd(t["dy"], out["codes3"], _L3, 3, dx=out["dx3"])
    lmbp.stepact_fwd(t["g"], "silu", _C4, 4, y=out["y4"], codes=out["codes4"])
    lmbp.stepact_bwd(t["dy"], out["codes4"], _L4, 4, dx=out["dx4"])
    if t["x"].dtype == torch.bfloat16:
        lmbp.linear_act_fwd(t["x"], t["w"], t["b"], act="gelu", y=out["yl"], codes=out["codesl"])


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_graph_replay_matches_eager(dtype):
    rows, p, f = 96, 1024, 2752
    t = {"x": T(inputs.normal((rows, p), 1.0, dtype, tensor_id=inputs.NORM_X)),
         "dz": T(inputs.normal((rows, p), 1.0, dtype, tensor_id=inputs.NORM_DZ)),
         "g": T(inputs.normal((rows, f), 2.0, dtype, tensor_id=inputs.ACT_X)),
         "dy": T(inputs.normal((rows, f), 1.0, dtype, tensor_id=inputs.ACT_DY)),
         "u": T(inputs.normal((rows, f), 1.0, dtype, tensor_id=inputs.ACT_U))}
    if dtype == "bf16":
        t["w"] = T(inputs.normal((f, p), p ** -0.5, "bf16", tensor_id=inputs.LIN_W))
        t["b"] = T(inputs.normal((f,), 0.1, "bf16", tensor_id=inputs.LIN_B))

    def alloc():
        e = lambda like: torch.empty_like(like)
        o = {"z": e(t["x"]), "rstd": torch.empty(rows, dtype=torch.float32, device=DEV),
             "y": e(t["g"]), "codes": torch.empty(lmbp.codes_words(rows * f), dtype=torch.int32, device=DEV),
             "dg": e(t["g"]), "dx": e(t["x"]), "h": e(t["g"]), "s": e(t["g"]),
             "codes2": torch.empty(lmbp.codes_words(rows * f), dtype=torch.int32, device=DEV),
             "dg2": e(t["g"]), "du2": e(t["g"]), "zl": e(t["x"]),
             "rstdl": torch.empty(rows, dtype=torch.float32, device=DEV), "dxl": e(t["x"]),
             "y3": e(t["g"]), "dx3": e(t["g"]), "y4": e(t["g"]), "dx4": e(t["g"]),
             "codes3": torch.empty(-(-rows * f // 10), dtype=torch.int32, device=DEV),
             "codes4": torch.empty(-(-rows * f // 8), dtype=torch.int32, device=DEV)}
        if dtype == "bf16":   # the fused linear layer is bf16 only
            o.update(yl=e(t["g"]), codesl=torch.empty(lmbp.codes_words(rows * f), dtype=torch.int32, device=DEV))
        return o

    eager = alloc()
    _step(t, eager)
    torch.cuda.synchronize()
    ref = {k: v.clone() for k, v in eager.items()}

    graphed = alloc()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):     # one eager pass on the capture stream first
        _step(t, graphed)
    torch.cuda.current_stream().wait_stream(side)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        _step(t, graphed)
    for replay in range(3):
        for v in graphed.values():    # poison the outputs so a replay that writes nothing fails
            v.view(torch.uint8).fill_(0xA5)
        g.replay()
        torch.cuda.synchronize()
        for k in ref:
            assert torch.equal(graphed[k].view(torch.uint8), ref[k].view(torch.uint8)), \
                f"replay {replay}: {k} differs from the eager result"
        _step(t, eager)               # eager work between replays
        torch.cuda.synchronize()
