"""bench.py on the GPU, run as its own process with a short step count: it prints one
JSON line with the fields of the benchmark contract, and its numbers agree with each
other (value = bytes per step / step time; the roofline fraction = achieved / peak)."""

import json
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.parametrize("flags", [[], ["--swiglu"], ["--workload", "vit_b_fp32", "--graph"]],
                         ids=["plain", "swiglu", "vit_fp32_graph"])
def test_bench_prints_one_contract_line(flags):
    print(f"[bench contract] bench.py --steps 5 --warmup 5 --no-cpu-baseline {' '.join(flags)}", flush=True)
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--steps", "5", "--warmup", "5",
                        "--no-cpu-baseline", *flags],
                       capture_output=True, text=True, timeout=110, cwd=ROOT)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [l for l in r.stdout.splitlines() if l.strip()]
    assert len(lines) == 1, r.stdout
    d = json.loads(lines[0])
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better",
                "scaling", "vs_baseline", "dtype", "data", "config", "roofline"):
        assert key in d, key
    assert d["n_gpus"] == 1 and d["steps"] == 5 and d["warmup"] == 5
    assert d["unit"] == "GB/s" and d["higher_is_better"] is True and d["data"] == "synthetic"
    assert "workload" in d["config"]
    assert d["launch"] == ("hip_graph" if "--graph" in flags else "eager")
    if "--workload" in flags:
        assert d["config"]["workload"] == flags[flags.index("--workload") + 1]
    step_bytes = d["config"]["bytes_per_step"]
    assert d["value"] == pytest.approx(step_bytes / (d["ms_per_step"] * 1e-3) / 1e9, rel=2e-3)
    rf = d["roofline"]
    assert rf["bound"] == "hbm" and rf["unit"] == "GB/s" and rf["peak"] == 8000.0
    assert rf["frac"] == pytest.approx(rf["achieved"] / rf["peak"], abs=1e-4)
    assert 0.3 < rf["frac"] < 1.0
    assert rf["kernel"] in d["per_kernel"]
    for rec in d["per_kernel"].values():   # the same-size plain copy is a streaming ceiling
        assert rec["copy_same_bytes_us"] > 0
        assert rec["copy_over_kernel"] == pytest.approx(rec["copy_same_bytes_us"] / rec["us"], abs=2e-3)
    # the metric's other ops, MS-LN and ReGELU2, on the ViT-B batch-64 bf16 shapes
    vit = d["pairs_vit_b_bs64_bf16"]
    assert set(vit) == {"msln", "regelu2"}
    for rec in vit.values():
        assert rec["GBps"] == pytest.approx(rec["bytes"] / ((rec["fwd_us"] + rec["bwd_us"]) * 1e-6) / 1e9, rel=2e-3)
        assert 0.2 < rec["pct_of_peak"] / 100 < 1.0
