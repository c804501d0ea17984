"""The GELU polynomial tables of the kernels (csrc/gelu_poly.h), evaluated on the host
in an fp32 emulation of the kernels' operation order, against the exact GELU of the
oracle. This checks the generated constants and the evaluation scheme (argument
mapping, clamping at T, folding of the quadratic term, the factor outside the
exponential); the kernels themselves are checked on the GPU.

Emulation: each fp32 operation is done in float64 and rounded to float32 once (a
fused multiply-add of fp32 operands is exact in float64 before that rounding, up to a
2^-53 relative term); the hardware exponential is taken as exact and flushes
subnormal results to zero, as the exponential unit does."""

import os
import re

import numpy as np

import oracle

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                      "paper_2406_16282_amd", "csrc", "gelu_poly.h")
NORMAL_MIN = 2.0 ** -126


def _hexf(s):
    return float.fromhex(s.rstrip("f"))


def read_table():
    text = open(HEADER).read()
    defs = {m.group(1): _hexf(m.group(2)) for m in re.finditer(r"#define (LMBP_GELU_\w+) (\S+)", text)}
    arrays = {}
    for m in re.finditer(r"kGelu(\w+)\[\d+\] = \{([^}]*)\}", text):
        arrays[m.group(1)] = np.array([_hexf(v.strip()) for v in m.group(2).split(",")], dtype=np.float32)
    return defs, arrays


def f32(v):
    return np.asarray(v, dtype=np.float64).astype(np.float32)


def fma(a, b, c):
    return f32(np.float64(a) * np.float64(b) + np.float64(c))


def exp2_flush(v):
    r = f32(np.exp2(np.float64(v)))
    return np.where(np.abs(r) < NORMAL_MIN, np.float32(0.0), r)


def horner(c, v):
    r = np.full_like(v, c[0])
    for k in c[1:]:
        r = fma(r, v, k)
    return r


def gelu_bf16_path(x, defs, arrays):
    x = f32(x)
    u = np.clip(f32(np.abs(x) * np.float64(np.float32(defs["LMBP_GELU_INV_T"]))), 0.0, 1.0).astype(np.float32)
    q = exp2_flush(horner(arrays["P8"], u))
    return fma(-u, q, np.maximum(x, 0.0))


def gelu_fp32_path(x, defs, arrays):
    x = f32(x)
    t = np.abs(x)
    T = np.float32(defs["LMBP_GELU_T"])
    v = fma(np.minimum(t, T), np.float32(defs["LMBP_GELU_2_OVER_T"]), -1.0)
    r = horner(arrays["R14"], v)
    hi = np.float32(0.72134752044448170368)
    lo = np.float32(0.72134752044448170368 - np.float64(hi))
    tc = np.minimum(t, np.float32(16.0))
    a_hi = f32(tc * -np.float64(hi))
    a_lo = fma(tc, -lo, fma(tc, -hi, -a_hi))
    k = np.rint(fma(tc, a_hi, r))
    f = f32(np.float64(fma(tc, a_hi, -k)) + np.float64(fma(tc, a_lo, r)))
    q = f32(np.ldexp(np.float64(exp2_flush(f)), k.astype(np.int64)))   # ldexp keeps subnormals
    return fma(-t, q, np.maximum(x, 0.0))


def _rel_err(y, x):
    ref = oracle.gelu(np.asarray(x, dtype=np.float64))
    m = np.abs(ref) >= NORMAL_MIN
    return np.max(np.abs(np.float64(y[m]) - ref[m]) / np.abs(ref[m])), ref


def test_bf16_path_on_every_bf16_value():
    defs, arrays = read_table()
    b = np.arange(0, 0x10000, dtype=np.uint32)
    x = (b << 16).view(np.float32)
    x = x[np.isfinite(x)]
    y = gelu_bf16_path(x, defs, arrays)
    err, ref = _rel_err(y, x)
    assert err < 2e-3, err                   # before bf16's own rounding (2^-9)
    assert np.all(np.isfinite(y))
    tiny = np.abs(ref) < NORMAL_MIN
    assert np.all(np.abs(y[tiny]) < NORMAL_MIN)
    # the bulk of the values (|x| < 5) to the accuracy that keeps bf16 rounding exact
    bulk = (np.abs(x) < 5.0) & (x != 0)
    assert _rel_err(y[bulk], x[bulk])[0] < 3e-5


def test_fp32_path_dense_and_tail():
    defs, arrays = read_table()
    x = np.concatenate([np.linspace(-14.0, 14.0, 400_001), np.linspace(-30.0, 30.0, 6001),
                        [1e4, -1e4, 3e38, -3e38, 1e-40, -1e-40, 0.0]]).astype(np.float32)
    y = gelu_fp32_path(x, defs, arrays)
    err, ref = _rel_err(y, x)
    assert err < 2e-6, err
    assert np.all(np.isfinite(y))
    assert np.all(np.abs(y[np.abs(ref) < NORMAL_MIN]) < NORMAL_MIN)


def test_domain_end_is_where_the_tail_leaves_the_normal_range():
    """Beyond T the kernels return max(x, 0) (up to a subnormal): t Q(t) must be below
    2^-126 there."""
    defs, _ = read_table()
    T = defs["LMBP_GELU_T"]
    assert abs(float(oracle.gelu(np.array([-T]))[0])) < NORMAL_MIN
    assert abs(float(oracle.gelu(np.array([-(T - 0.5)]))[0])) > NORMAL_MIN
