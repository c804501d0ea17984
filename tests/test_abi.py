"""C ABI checks that need no GPU: the library loads, exports every declared entry
point, and rejects invalid calls on the host before any launch."""

import ctypes
import math
import os
import re

import pytest

import paper_2406_16282_amd as lmbp
from paper_2406_16282_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "lmbp.h")

# Fake device addresses: every call below fails validation before anything is
# launched or dereferenced.
P = 0x7F0000000000


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[a-z_0-9]+\s*\*?\s*([a-z_0-9]+)\s*\(", text, flags=re.M)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(B.LIB_PATH):
        pytest.fail("liblmbp.so is not built; run __graft_entry__.build()")
    return lmbp.lib()


def test_every_declared_symbol_is_exported(L):
    names = declared_functions()
    assert set(B.ACT_OPS + B.NORM_OPS + B.GLU_OPS) <= set(names)
    for name in names:
        assert hasattr(L, name), name


def test_codes_bytes(L):
    assert [L.lmbp_codes_bytes(n) for n in (-5, 0, 1, 15, 16, 17, 32, 33)] == [0, 0, 4, 4, 4, 8, 8, 12]
    assert L.lmbp_codes_bytes(90177536) == 90177536 // 4


def test_strerror(L):
    for st in range(5):
        assert len(B.strerror(st)) > 3
    assert B.strerror(99) == "unknown status"


@pytest.mark.parametrize("op", B.ACT_OPS)
def test_activation_errors(L, op):
    f = getattr(L, op)
    s = None
    assert f(7, 16, P, P + 4096, P + 8192, s) == B.EDTYPE
    assert f(B.FP32, -1, P, P + 4096, P + 8192, s) == B.EINVAL
    assert f(B.FP32, 0, P, P + 4096, P + 8192, s) == B.OK          # no-op
    assert f(B.FP32, 0, None, None, None, s) == B.OK
    assert f(B.FP32, 16, None, P + 4096, P + 8192, s) == B.EINVAL
    assert f(B.FP32, 16, P, None, P + 8192, s) == B.EINVAL
    assert f(B.FP32, 16, P, P + 4096, None, s) == B.EINVAL
    assert f(B.FP32, 16, P + 2, P + 4096, P + 8192, s) == B.EINVAL  # not element aligned
    assert f(B.BF16, 16, P + 1, P + 4096, P + 8192, s) == B.EINVAL
    assert f(B.FP32, 16, P, P + 4096, P + 8194, s) == B.EINVAL     # codes not 4-byte aligned
    assert f(B.FP32, 16, P, P + 32, P + 8192, s) == B.EOVERLAP     # partial overlap of tensors
    assert f(B.FP32, 16, P, P + 4096, P + 60, s) == B.EOVERLAP     # codes inside the first tensor
    assert f(B.FP32, 16, P, P + 4096, P + 4096, s) == B.EOVERLAP   # codes on the second tensor
    assert f(B.FP32, 1 << 61, P, P + 4096, P + 8192, s) == B.EINVAL


@pytest.mark.parametrize("op", ["msln_fwd", "msrms_fwd"])
def test_norm_fwd_errors(L, op):
    f = getattr(L, op)
    s = None
    assert f(9, 4, 8, 1e-5, P, P + 4096, P + 8192, s) == B.EDTYPE
    assert f(B.FP32, -1, 8, 1e-5, P, P + 4096, P + 8192, s) == B.EINVAL
    assert f(B.FP32, 4, -8, 1e-5, P, P + 4096, P + 8192, s) == B.EINVAL
    assert f(B.FP32, 4, 0, 1e-5, P, P + 4096, P + 8192, s) == B.EINVAL
    assert f(B.FP32, 0, 8, 1e-5, P, P + 4096, P + 8192, s) == B.OK
    for eps in (0.0, -1e-5, math.inf, math.nan):
        assert f(B.FP32, 4, 8, eps, P, P + 4096, P + 8192, s) == B.EINVAL
    assert f(B.FP32, 4, 8, 1e-5, None, P + 4096, P + 8192, s) == B.EINVAL
    assert f(B.FP32, 4, 8, 1e-5, P, P + 4096, P + 8194, s) == B.EINVAL  # rstd misaligned
    assert f(B.BF16, 4, 8, 1e-5, P + 1, P + 4096, P + 8192, s) == B.EINVAL
    assert f(B.FP32, 4, 8, 1e-5, P, P + 64, P + 8192, s) == B.EOVERLAP   # x/z partial overlap
    assert f(B.FP32, 4, 8, 1e-5, P, P + 4096, P + 100, s) == B.EOVERLAP  # rstd inside x
    assert f(B.FP32, 4, 8, 1e-5, P, P + 4096, P + 4096, s) == B.EOVERLAP # rstd on z


@pytest.mark.parametrize("op", ["msln_bwd", "msrms_bwd"])
def test_norm_bwd_errors(L, op):
    f = getattr(L, op)
    s = None
    dz, z, r, dx = P, P + 4096, P + 8192, P + 12288
    assert f(3, 4, 8, dz, z, r, dx, s) == B.EDTYPE
    assert f(B.FP32, 4, 0, dz, z, r, dx, s) == B.EINVAL
    assert f(B.FP32, 0, 8, dz, z, r, dx, s) == B.OK
    assert f(B.FP32, 4, 8, dz, z, r, None, s) == B.EINVAL
    assert f(B.FP32, 4, 8, dz, z, r + 2, dx, s) == B.EINVAL
    assert f(B.FP32, 4, 8, dz, z, r, z, s) == B.EOVERLAP          # dx on z is not allowed
    assert f(B.FP32, 4, 8, dz, z, r, dz + 4, s) == B.EOVERLAP     # partial overlap with dz
    assert f(B.FP32, 4, 8, dz, z, dz + 16, dx, s) == B.EOVERLAP   # rstd inside dz


def test_swiglu_errors(L):
    f, b = L.reswiglu2_fwd, L.reswiglu2_bwd
    g, u, h, s, c = P, P + 4096, P + 8192, P + 12288, P + 16384
    assert f(5, 16, g, u, h, s, c, None) == B.EDTYPE
    assert f(B.BF16, -1, g, u, h, s, c, None) == B.EINVAL
    assert f(B.BF16, 0, g, u, h, s, c, None) == B.OK
    assert f(B.BF16, 16, g, u, h, None, c, None) == B.EINVAL
    assert f(B.BF16, 16, g + 1, u, h, s, c, None) == B.EINVAL
    assert f(B.BF16, 16, g, g + 8, h, s, c, None) == B.EOVERLAP    # g and u overlap
    assert f(B.BF16, 16, g, u, h, g, c, None) == B.EOVERLAP        # s on an input
    assert f(B.BF16, 16, g, u, h, s, s + 4, None) == B.EOVERLAP    # codes inside s
    assert f(B.BF16, 16, g, u, h, h + 2, c, None) == B.EOVERLAP    # s overlaps h
    dh, dg, du = P, P + 20480, P + 24576
    assert b(B.BF16, -3, dh, u, s, c, dg, du, None) == B.EINVAL
    assert b(B.BF16, 16, dh, u, s, c, dg, None, None) == B.EINVAL
    assert b(B.BF16, 16, dh, u, s, c, s, du, None) == B.EOVERLAP      # dg on s
    assert b(B.BF16, 16, dh, u, s, c, dg, dh, None) == B.EOVERLAP     # du on dh
    assert b(B.BF16, 16, dh, u, s, c, dg, dg, None) == B.EOVERLAP     # dg and du alias
    assert b(B.BF16, 16, dh, u, s, dg + 4, dg, du, None) == B.EOVERLAP


def test_linear_act_errors(L):
    f = L.linear_act_fwd
    G = B.ACT_GELU
    # m = 4, n = 32, k = 16: x 128 B, w 1024 B, bias 64 B, y / z 256 B, codes 32 B
    x, w, bias, y, c, z = P, P + 4096, P + 8192, P + 12288, P + 16384, P + 20480
    assert f(G, B.FP32, 4, 32, 16, x, w, bias, y, c, z, None) == B.EDTYPE
    assert f(G, 7, 4, 32, 16, x, w, bias, y, c, z, None) == B.EDTYPE
    assert f(9, B.BF16, 4, 32, 16, x, w, bias, y, c, z, None) == B.EINVAL
    assert f(G, B.BF16, -1, 32, 16, x, w, bias, y, c, z, None) == B.EINVAL
    assert f(G, B.BF16, 4, 24, 16, x, w, bias, y, c, z, None) == B.EINVAL     # n % 16
    assert f(G, B.BF16, 4, 32, 12, x, w, bias, y, c, z, None) == B.EINVAL     # k % 8
    assert f(G, B.BF16, 4, 32, (1 << 21) + 8, x, w, bias, y, c, z, None) == B.EINVAL  # k limit
    assert f(G, B.BF16, 0, 32, 16, x, w, bias, y, c, z, None) == B.OK         # empty
    assert f(G, B.BF16, 4, 0, 16, x, w, bias, y, c, z, None) == B.OK
    assert f(G, B.BF16, 4, 32, 16, x, w, bias, None, c, z, None) == B.EINVAL
    assert f(G, B.BF16, 4, 32, 16, None, w, bias, y, c, z, None) == B.EINVAL
    assert f(G, B.BF16, 4, 32, 16, x + 8, w, bias, y, c, z, None) == B.EINVAL   # 16-byte alignment
    assert f(G, B.BF16, 4, 32, 16, x, w, bias, y, c, z + 2, None) == B.EINVAL
    assert f(G, B.BF16, 4, 32, 16, x, w, bias + 1, y, c, z, None) == B.EINVAL
    assert f(G, B.BF16, 4, 32, 16, x, w, bias, y, c, y + 16, None) == B.EOVERLAP  # z overlaps y
    assert f(G, B.BF16, 4, 32, 16, x, w, bias, y, x + 64, z, None) == B.EOVERLAP  # codes on x
    assert f(G, B.BF16, 4, 32, 16, x, w, bias, w, c, z, None) == B.EOVERLAP       # y on w
    assert f(G, B.BF16, 4, 32, 16, x, w, bias, y, c, bias - 16, None) == B.EOVERLAP


def test_linear_swiglu_errors(L):
    f = L.linear_swiglu_fwd
    x, wg, wu, h, s, u, c, g = (P + 4096 * i for i in range(8))
    assert f(B.FP32, 4, 32, 16, x, wg, wu, h, s, u, c, g, None) == B.EDTYPE
    assert f(B.BF16, -1, 32, 16, x, wg, wu, h, s, u, c, g, None) == B.EINVAL
    assert f(B.BF16, 4, 24, 16, x, wg, wu, h, s, u, c, g, None) == B.EINVAL      # n % 16
    assert f(B.BF16, 4, 32, 12, x, wg, wu, h, s, u, c, g, None) == B.EINVAL      # k % 8
    assert f(B.BF16, 0, 32, 16, x, wg, wu, h, s, u, c, g, None) == B.OK
    assert f(B.BF16, 4, 32, 16, x, wg, wu, h, None, u, c, g, None) == B.EINVAL
    assert f(B.BF16, 4, 32, 16, x, None, wu, h, s, u, c, g, None) == B.EINVAL
    assert f(B.BF16, 4, 32, 16, x, wg, wu + 8, h, s, u, c, g, None) == B.EINVAL   # alignment
    assert f(B.BF16, 4, 32, 16, x, wg, wu, h, h, u, c, g, None) == B.EOVERLAP     # s on h
    assert f(B.BF16, 4, 32, 16, x, wg, wu, h, s, wu, c, g, None) == B.EOVERLAP    # u on w_up
    assert f(B.BF16, 4, 32, 16, x, wg, wu, h, s, u, c, c - 16, None) == B.EOVERLAP  # g on codes


def test_msrms_linear_act_errors(L):
    f = L.msrms_linear_act_fwd
    G = B.ACT_SILU
    # m = 4, n = 32, k = 16: x / z 128 B, w 1024 B, bias 64 B, y 256 B, codes 32 B, rstd 16 B
    x, w, bias, y, c, z, r, a = (P + 4096 * i for i in range(8))
    assert f(G, B.FP32, 4, 32, 16, 1e-5, x, w, bias, y, c, None, z, r, None) == B.EDTYPE
    assert f(9, B.BF16, 4, 32, 16, 1e-5, x, w, bias, y, c, None, z, r, None) == B.EINVAL
    assert f(G, B.BF16, 4, 32, 16, 0.0, x, w, bias, y, c, None, z, r, None) == B.EINVAL            # eps
    assert f(G, B.BF16, 4, 32, 16, float("nan"), x, w, bias, y, c, None, z, r, None) == B.EINVAL
    assert f(G, B.BF16, 4, 24, 16, 1e-5, x, w, bias, y, c, None, z, r, None) == B.EINVAL           # n % 16
    assert f(G, B.BF16, 4, 32, 12, 1e-5, x, w, bias, y, c, None, z, r, None) == B.EINVAL           # k % 8
    assert f(G, B.BF16, 4, 32, 0, 1e-5, x, w, bias, y, c, None, z, r, None) == B.EINVAL            # no row
    assert f(G, B.BF16, 0, 32, 16, 1e-5, x, w, bias, y, c, None, z, r, None) == B.OK               # empty
    assert f(G, B.BF16, 4, 32, 16, 1e-5, x, w, bias, y, c, None, None, r, None) == B.EINVAL        # z required
    assert f(G, B.BF16, 4, 32, 16, 1e-5, x, w, bias, y, c, None, z, None, None) == B.EINVAL        # rstd required
    assert f(G, B.BF16, 4, 32, 16, 1e-5, x, w, bias, y, c, None, z + 8, r, None) == B.EINVAL       # alignment
    assert f(G, B.BF16, 4, 32, 16, 1e-5, x, w, bias, y, c, None, z, r + 2, None) == B.EINVAL
    assert f(G, B.BF16, 4, 32, 16, 1e-5, x, w, bias, y, c, None, x, r, None) == B.EOVERLAP         # z on x
    assert f(G, B.BF16, 4, 32, 16, 1e-5, x, w, bias, y, c, None, z, y + 64, None) == B.EOVERLAP    # rstd on y
    assert f(G, B.BF16, 4, 32, 16, 1e-5, x, w, bias, y, c, None, z, w, None) == B.EOVERLAP         # rstd on w
    assert f(G, B.BF16, 4, 32, 16, 1e-5, x, w, bias, y, c, a + 2, z, r, None) == B.EINVAL          # pre alignment
    assert f(G, B.BF16, 4, 32, 16, 1e-5, x, w, bias, y, c, y + 64, z, r, None) == B.EOVERLAP       # pre on y


def test_msrms_linear_swiglu_errors(L):
    f = L.msrms_linear_swiglu_fwd
    x, wg, wu, h, s, u, c, z, r = (P + 4096 * i for i in range(9))
    g = None
    assert f(B.FP32, 4, 32, 16, 1e-5, x, wg, wu, h, s, u, c, g, z, r, None) == B.EDTYPE
    assert f(B.BF16, 4, 32, 16, -1.0, x, wg, wu, h, s, u, c, g, z, r, None) == B.EINVAL
    assert f(B.BF16, 4, 32, 12, 1e-5, x, wg, wu, h, s, u, c, g, z, r, None) == B.EINVAL
    assert f(B.BF16, 0, 32, 16, 1e-5, x, wg, wu, h, s, u, c, g, z, r, None) == B.OK
    assert f(B.BF16, 4, 32, 16, 1e-5, x, wg, wu, h, s, u, c, g, None, r, None) == B.EINVAL
    assert f(B.BF16, 4, 32, 16, 1e-5, x, wg, wu, h, s, u, c, g, h, r, None) == B.EOVERLAP      # z on h
    assert f(B.BF16, 4, 32, 16, 1e-5, x, wg, wu, h, s, u, c, g, z, c, None) == B.EOVERLAP      # rstd on codes
    assert f(B.BF16, 4, 32, 16, 1e-5, x, wg, wu, h, s, u, c, u + 16, z, r, None) == B.EOVERLAP  # g on u
    assert f(B.BF16, 4, 32, 16, 1e-5, x, wg, wu, h, s, u, c, P + 4096 * 9 + 2, z, r, None) == B.EINVAL


def test_copy_errors(L):
    assert L.lmbp_copy(P, P + 4096, -1, None) == B.EINVAL
    assert L.lmbp_copy(P, P + 4096, 0, None) == B.OK
    assert L.lmbp_copy(P + 8, P + 4096, 64, None) == B.EINVAL
    assert L.lmbp_copy(P, P + 32, 64, None) == B.EOVERLAP


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(B, "_lib", None)
    monkeypatch.setattr(B, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(RuntimeError, match="missing"):
        B.lib()


def test_binding_rejects_cpu_tensors(L):
    import torch
    with pytest.raises(ValueError):
        lmbp.resilu2_fwd(torch.zeros(16, dtype=torch.bfloat16))


def test_stepact_errors(L):
    import ctypes
    t3 = (ctypes.c_double * 3)(-1.0, 0.0, 1.0)
    bad = (ctypes.c_double * 3)(-1.0, 1.0, 0.5)       # not increasing
    nan = (ctypes.c_double * 3)(-1.0, float("nan"), 1.0)
    lv4 = (ctypes.c_double * 4)(0.0, 0.2, 0.7, 1.0)
    f, b = L.stepact_fwd, L.stepact_bwd
    x, y, c = P, P + 4096, P + 8192
    assert f(0, 2, t3, 7, 16, x, y, c, None) == B.EDTYPE
    assert f(0, 5, t3, B.BF16, 16, x, y, c, None) == B.EINVAL     # k = 5 not supported
    assert f(0, 0, t3, B.BF16, 16, x, y, c, None) == B.EINVAL     # nor k = 0
    t7 = (ctypes.c_double * 7)(-3.0, -2.0, -1.0, 0.0, 1.0, 2.0, 3.0)
    assert f(0, 3, t7, B.BF16, 0, x, y, c, None) == B.OK          # k = 3: seven thresholds
    assert b(3, (ctypes.c_double * 8)(*range(8)), B.BF16, 0, x, c, y, None) == B.OK
    assert f(5, 2, t3, B.BF16, 16, x, y, c, None) == B.EINVAL     # unknown activation
    assert f(0, 2, None, B.BF16, 16, x, y, c, None) == B.EINVAL
    assert f(0, 2, bad, B.BF16, 16, x, y, c, None) == B.EINVAL
    assert f(0, 2, nan, B.BF16, 16, x, y, c, None) == B.EINVAL
    assert f(0, 2, t3, B.BF16, 0, x, y, c, None) == B.OK
    assert f(0, 2, t3, B.BF16, 16, x, x + 2, c, None) == B.EOVERLAP
    assert b(2, None, B.BF16, 16, x, c, y, None) == B.EINVAL
    assert b(2, lv4, B.BF16, 16, x, x + 4, y, None) == B.EOVERLAP
    # words of floor(32/k) codes: 2, 3, 4 (10 per word), 5 words for 33 elements; k = 5: 0
    assert [L.lmbp_stepact_codes_bytes(k, 33) for k in (1, 2, 3, 4, 5)] == [8, 12, 16, 20, 0]
