"""Build liblmbp.so for gfx950 with hipcc (in-tree, next to this file).

Each HIP source is compiled to an object in parallel, then linked into one shared
library. Device code is built with packed-FP32 instruction selection disabled.
"""

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD_DIR = os.path.join(ROOT, "_build")
LIB_PATH = os.path.join(HERE, "liblmbp.so")
SOURCES = ("lmbp_api.hip", "act_kernels.hip", "norm_kernels.hip", "stepact_kernels.hip",
           "linear_kernels.hip")
ARCH = "gfx950"

COMMON_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-command-line-argument",
    "-I", INCLUDE, "-I", CSRC,
]


def _hipcc():
    exe = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(exe):
        raise RuntimeError("hipcc not found; the ROCm toolchain is required to build liblmbp")
    return exe


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    # hipcc's host pass does not know the packed-fp32 target feature and says so; that
    # line is expected and dropped from the log.
    out = "\n".join(l for l in r.stdout.splitlines() if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}\n{out}")
    return out


def build(verbose=False, defines=(), lib_path=LIB_PATH, build_dir=BUILD_DIR):
    """Compile and link the library. `defines` are extra -D macros (tuning knobs
    of the kernel sources); the defaults produce the shipped configuration."""
    hipcc = _hipcc()
    os.makedirs(build_dir, exist_ok=True)
    flags = COMMON_FLAGS + [f"-D{d}" for d in defines]
    objs = []
    cmds = []
    for src in SOURCES:
        obj = os.path.join(build_dir, src.replace(".hip", ".o"))
        objs.append(obj)
        cmds.append([hipcc, *flags, "-c", os.path.join(CSRC, src), "-o", obj])
    with cf.ThreadPoolExecutor(max_workers=len(cmds)) as ex:
        logs = list(ex.map(_run, cmds))
    tmp = lib_path + ".tmp"
    logs.append(_run([hipcc, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]))
    os.replace(tmp, lib_path)
    if verbose:
        for l in logs:
            if l.strip():
                print(l)
    return lib_path


if __name__ == "__main__":
    print(build(verbose=True))
    sys.exit(0)
