"""Host-side parts of bench.py, checked without a GPU: the algorithmic byte counts it
divides by (written out here from the per-element accounting of each kernel), and the
refusal of more than one GPU."""

import os
import subprocess
import sys

import bench
from paper_2406_16282_amd import inputs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_llama7b_step_bytes():
    # MS-RMSNorm on [8192, 4096] bf16 (x in, z out, 4 B of rstd per row; backward dz and
    # z in, dx out) and ReSiLU2 on [8192, 11008] bf16 (x in, y out, 2 bits per element;
    # backward dy and codes in, dx out).
    w = inputs.WORKLOADS["llama7b_swiglu_bf16"]
    nb = bench.algorithmic_bytes(w)
    n_norm, n_act = 8192 * 4096, 8192 * 11008
    assert nb == {
        "msrms_fwd": 2 * 2 * n_norm + 4 * 8192,
        "resilu2_fwd": 2 * 2 * n_act + n_act // 4,
        "resilu2_bwd": 2 * 2 * n_act + n_act // 4,
        "msrms_bwd": 3 * 2 * n_norm + 4 * 8192,
    }
    assert sum(nb.values()) == 1_102_118_912


def test_fused_swiglu_step_bytes():
    # g and u in, h and s out, codes out; dh, u, s and codes in, dg and du out.
    w = inputs.WORKLOADS["llama7b_swiglu_bf16"]
    nb = bench.algorithmic_bytes(w, swiglu=True)
    n = 8192 * 11008
    assert nb["reswiglu2_fwd"] == 4 * 2 * n + n // 4
    assert nb["reswiglu2_bwd"] == 5 * 2 * n + n // 4
    assert sum(nb.values()) == 2_003_894_272


def test_codes_round_up_to_whole_words():
    # A ragged activation count still stores whole 32-bit words of 16 codes.
    w = inputs.WORKLOADS["vit_b_fp32"]
    n = w.act.rows * w.act.cols
    nb = bench.algorithmic_bytes(w)
    assert nb["regelu2_fwd"] == 2 * 4 * n + 4 * ((n + 15) // 16)


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_unknown_workload_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--workload", "no_such_shape",
                        "--no-cpu-baseline"], capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert r.returncode != 0 and "--workload must be one of" in r.stderr and r.stdout == ""
