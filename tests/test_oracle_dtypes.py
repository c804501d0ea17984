"""Pins of the oracle's storage decoding and rounding."""

import numpy as np

import oracle
import pins


def test_bf16_decode_known_patterns():
    pats = np.array([0x3F80, 0xC040, 0x0001, 0x7F7F, 0x8000, 0x3E80], dtype=np.uint16)
    want = [1.0, -3.0, 2.0 ** -133, (2 - 2 ** -7) * 2.0 ** 127, -0.0, 0.25]
    got = oracle.decode(pats, "bf16")
    assert list(got) == want
    assert np.signbit(got[4])


def test_bf16_rounding_against_exact_rationals():
    assert pins.pin_bf16_rounding(oracle.round_to_dtype) == 0


def test_encode_decode_round_trip():
    g = np.random.default_rng(0)
    x = g.normal(0, 3, 1000)
    for dt in oracle.DTYPES:
        r = oracle.round_to_dtype(x, dt)
        assert np.array_equal(oracle.decode(oracle.encode(x, dt), dt), r)
        assert np.array_equal(oracle.round_to_dtype(r, dt), r)


def test_fp32_rounding_is_nearest():
    g = np.random.default_rng(1)
    x = g.normal(0, 3, 1000)
    r = oracle.round_to_dtype(x, "fp32").astype(np.float32)
    up = np.nextafter(r, np.float32(np.inf)).astype(np.float64)
    dn = np.nextafter(r, np.float32(-np.inf)).astype(np.float64)
    d = np.abs(x - r.astype(np.float64))
    assert np.all(d <= np.abs(x - up)) and np.all(d <= np.abs(x - dn))
