"""Comparison rules between the HIP path and the CPU oracle.

Tolerances (stated for the method's floating-point outputs):
  rtol = 1e-5 for fp32 tensors and for the fp32 norm statistic rstd,
  rtol = 1e-2 for bf16 tensors.

Mixed rule (all float outputs): |got - ref| <= rtol * (|ref| + s_row), where s_row
is the root mean square of the oracle output over the element's row. A pure
elementwise relative test cannot hold for outputs that cancel to nearly zero
(norm outputs and gradients), even for an exact fp32 evaluation; the row scale is
the natural size against which their rounding is measured.

Norm backward: dx = rstd * (dz - mean(dz) - z * mean(z * dz)) (Alg. 2, Alg. 3) is a
projection of rstd * dz, and its rounding is bounded relative to the size of the
terms it combines, rstd * rms(dz), not relative to its result: for rows where the
projection nearly annihilates dz (a LayerNorm row of two elements has z = +-1 up
to eps, so dx is of order eps) the output RMS is no measure of the arithmetic.
There s_row is max(rms(ref), rstd * rms(dz)) (``norm_grad_scale``).

Strict rules (activations): the forward value is within rtol relative for every
element with |ref| >= 2^-126, the smallest normal fp32 / bf16 magnitude (below it
the result is subnormal in both storage formats and only the mixed rule applies);
the backward value is within rtol relative everywhere and is exactly +-0 where the
code is 0. Products of two storage values (the SwiGLU gradients dg = dh u slope and
du = dh s) can fall below the smallest normal and below bf16's subnormal range, so for
them the strict rule applies where |ref| >= 2^-126, like the forward's.

Integer outputs (codes) are compared bit for bit.
"""

import numpy as np


def rtol_for(dtype):
    return 1e-5 if dtype == "fp32" else 1e-2


def _rows2d(a):
    a = np.asarray(a, dtype=np.float64)
    return a.reshape(1, -1) if a.ndim == 1 else a.reshape(-1, a.shape[-1])


def norm_grad_scale(dz, rstd):
    """Per-row size rstd * rms(dz) of the terms of a norm backward."""
    d = _rows2d(dz)
    return np.asarray(rstd, dtype=np.float64).reshape(-1, 1) * np.sqrt(np.mean(d * d, axis=1, keepdims=True))


def assert_mixed(got, ref, rtol, what, row_scale=None):
    g, r = _rows2d(got), _rows2d(ref)
    assert g.shape == r.shape, f"{what}: shape {g.shape} vs {r.shape}"
    assert np.all(np.isfinite(g)), f"{what}: non-finite values"
    s = np.sqrt(np.mean(r * r, axis=1, keepdims=True))
    if row_scale is not None:
        s = np.maximum(s, np.asarray(row_scale, dtype=np.float64).reshape(-1, 1))
    err = np.abs(g - r)
    lim = rtol * (np.abs(r) + s)
    bad = err > lim
    if bad.any():
        i = np.argwhere(bad)[0]
        ratio = float(np.max(err / np.where(lim > 0, lim, np.inf)))
        raise AssertionError(
            f"{what}: {int(bad.sum())} of {bad.size} elements outside the mixed tolerance "
            f"(rtol {rtol}); first at {tuple(i)}: got {g[tuple(i)]!r} ref {r[tuple(i)]!r}; "
            f"worst err/limit {ratio:.3g}")
    return float(np.max(err / np.maximum(lim, 1e-300)))


NORMAL_MIN = 2.0 ** -126


def assert_rel(got, ref, rtol, what, floor=NORMAL_MIN):
    g = np.asarray(got, dtype=np.float64).reshape(-1)
    r = np.asarray(ref, dtype=np.float64).reshape(-1)
    m = (np.abs(r) >= floor) & (r != 0)
    err = np.abs(g[m] - r[m]) / np.abs(r[m])
    zero = (r == 0) & (np.abs(r) >= floor)
    if np.any(g[zero] != 0):
        idx = np.flatnonzero(zero)[np.flatnonzero(g[zero] != 0)[0]]
        raise AssertionError(f"{what}: expected exact zero at flat index {idx}, got {g[idx]!r}")
    if err.size and err.max() > rtol:
        k = int(np.argmax(err))
        idx = np.flatnonzero(m)[k]
        raise AssertionError(f"{what}: relative error {err[k]:.3g} > {rtol} at flat index {idx}: "
                             f"got {g[idx]!r} ref {r[idx]!r}")
    return float(err.max()) if err.size else 0.0


def assert_codes_equal(got_words, ref_words, what):
    g = np.asarray(got_words).view(np.uint32).reshape(-1)
    r = np.asarray(ref_words).view(np.uint32).reshape(-1)
    assert g.size == r.size, f"{what}: {g.size} words vs {r.size}"
    diff = np.flatnonzero(g != r)
    if diff.size:
        k = int(diff[0])
        raise AssertionError(f"{what}: {diff.size} code words differ; first word {k}: "
                             f"got {int(g[k]):#010x} ref {int(r[k]):#010x}")


def bf16_ulp_distance(got_bits, ref64):
    """Distance in bf16 steps between stored bf16 values and the oracle's correctly
    rounded value (same-sign finite values; sign-magnitude ordering)."""
    from oracle import encode
    def key(b):
        b = np.asarray(b, dtype=np.uint16).astype(np.int64)
        mag = b & 0x7FFF
        return np.where(b & 0x8000, -mag, mag)
    return np.abs(key(got_bits) - key(encode(ref64, "bf16")))
