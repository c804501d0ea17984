"""Pins of the oracle's general k-bit family and ReGELU2-d."""

import numpy as np
import pytest

import oracle
from oracle import variants as V
import pins


def test_regelu2d_constants_match_appendix_i():
    g = pins.read_golden_constants()
    assert list(V.REGELU2D_A) == g["regelu2d_a"]
    assert list(V.REGELU2D_C) == g["regelu2d_c"]


def test_k2_family_equals_the_k2_oracle():
    x = np.random.default_rng(0).normal(0, 3, 1000)
    for a, c in ((oracle.GELU_A, oracle.GELU_C), (oracle.SILU_A, oracle.SILU_C)):
        assert np.allclose(V.relu_family(x, a, c), oracle.relu_combination(x, a, c), atol=1e-14)
        assert np.array_equal(V.family_code(x, c), oracle.segment_code(x, c))
        assert np.array_equal(V.family_levels(a), oracle.derivative_levels(a))
        assert np.array_equal(V.pack_bits(V.family_code(x, c), 2), oracle.pack_codes(oracle.segment_code(x, c)))


@pytest.mark.parametrize("bits", [1, 2, 4])
def test_levels_are_slopes_for_every_k(bits):
    r = np.random.default_rng(bits)
    m = (1 << bits) - 1
    c = np.sort(r.uniform(-4, 4, m))
    a = list(r.normal(0, 0.5, m - 1))
    assert pins.pin_levels_fd(lambda x, a_, c_: V.relu_family(x, a_, c_), V.family_levels,
                              V.family_code, a, c) < 1e-8


@pytest.mark.parametrize("bits", [1, 2, 4])
def test_pack_round_trip_and_layout(bits):
    per = 32 // bits
    r = np.random.default_rng(7)
    for n in (1, per - 1, per, per + 1, 1000):
        codes = r.integers(0, 1 << bits, n).astype(np.uint8)
        w = V.pack_bits(codes, bits)
        assert w.size == V.words_for(bits, n)
        assert np.array_equal(V.unpack_bits(w, bits, n), codes)
    codes = np.zeros(per, dtype=np.uint8)
    codes[1] = 1
    assert int(V.pack_bits(codes, bits)[0]) == 1 << bits


def test_regelu2d_levels_match_gelu_derivative_roughly():
    # ReGELU2-d approximates GELU' directly: on each segment the level lies between the
    # derivative's values at the segment ends (a check of the reading, not of digits).
    from scipy.stats import norm
    d = lambda x: norm.cdf(x) + x * norm.pdf(x)
    lv = V.family_levels(V.REGELU2D_A)
    c = V.REGELU2D_C
    assert d(-6) - 1e-3 < lv[0] < d(c[0]) + 1e-3
    assert d(c[0]) < lv[1] < d(c[1]) and d(c[1]) < lv[2] < d(c[2]) and d(c[2]) < lv[3] < 1.13
