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


@pytest.mark.parametrize("bits", [1, 2, 3, 4])
def test_levels_are_slopes_for_every_k(bits):
    r = np.random.default_rng(bits)
    m = (1 << bits) - 1
    c = np.sort(r.uniform(-4, 4, m))
    a = list(r.normal(0, 0.5, m - 1))
    assert pins.pin_levels_fd(lambda x, a_, c_: V.relu_family(x, a_, c_), V.family_levels,
                              V.family_code, a, c) < 1e-8


@pytest.mark.parametrize("bits", [1, 2, 3, 4])
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


def test_three_bit_layout_by_hand():
    """k = 3: ten codes per word at bits 3j .. 3j + 2, top two bits zero, next word for
    the eleventh code (written out bit by bit, independent of pack_bits)."""
    codes = np.array([1, 2, 3, 4, 5, 6, 7, 0, 7, 6, 5], dtype=np.uint8)
    w0 = sum(int(c) << (3 * j) for j, c in enumerate(codes[:10]))
    assert list(V.pack_bits(codes, 3)) == [w0, 5]
    assert int(V.pack_bits(np.full(10, 7, dtype=np.uint8), 3)[0]) == 0x3FFFFFFF
    assert V.words_for(3, 10) == 1 and V.words_for(3, 11) == 2


def test_three_bit_family_codes_brute_force():
    """k = 3 (7 biases, 8 slopes): codes count the biases below x, per element."""
    r = np.random.default_rng(33)
    c = np.sort(r.uniform(-4, 4, 7))
    x = r.normal(0, 3, 2000)
    want = np.array([sum(1 for ci in c if xi > ci) for xi in x], dtype=np.uint8)
    assert np.array_equal(V.family_code(x, c), want)
    words = V.pack_bits(want, 3)
    assert np.array_equal(V.unpack_bits(words, 3, x.size), want)


def _random_table(bits, seed):
    r = np.random.default_rng(100 + seed)
    m = (1 << bits) - 1
    c = np.sort(r.uniform(-4, 4, m))
    while m > 1 and np.min(np.diff(c)) < 1e-2:
        c = np.sort(r.uniform(-4, 4, m))
    return list(r.normal(0, 0.5, m - 1)), list(c)


@pytest.mark.parametrize("act", ["gelu", "silu"])
@pytest.mark.parametrize("bits", [1, 2, 3, 4])
def test_stepact_composed_against_torch_and_fd_slopes(bits, act):
    a, c = _random_table(bits, bits)
    assert pins.pin_stepact_fd(V.stepact_fwd, V.stepact_bwd, V.relu_family, a, c, bits, act) < 1e-8


@pytest.mark.parametrize("table", ["gelu", "silu", "regelu2d"])
def test_stepact_composed_with_paper_tables(table):
    a, c, act = {"gelu": (oracle.GELU_A, oracle.GELU_C, "gelu"),
                 "silu": (oracle.SILU_A, oracle.SILU_C, "silu"),
                 "regelu2d": (V.REGELU2D_A, V.REGELU2D_C, "gelu")}[table]
    assert pins.pin_stepact_fd(V.stepact_fwd, V.stepact_bwd, V.relu_family, list(a), list(c), 2,
                               act) < 1e-8


@pytest.mark.parametrize("bits", [1, 2, 3, 4])
def test_stepact_words_against_a_bitwise_loop(bits):
    _, c = _random_table(bits, 20 + bits)
    assert pins.pin_stepact_words_brute(V.stepact_fwd, c, bits) == 0


def test_stepact_k2_is_byte_equal_to_the_dedicated_k2_oracle():
    """With Appendix E's tables and k = 2, the table-driven composition must give the
    same values, the same words and the same gradients as ReGELU2 / ReSiLU2."""
    r = np.random.default_rng(5)
    x = np.concatenate([r.normal(0, 3, 4001), np.array(oracle.GELU_C), np.array(oracle.SILU_C)])
    dy = r.normal(size=x.size)
    for act, a, c, fwd, bwd in (("gelu", oracle.GELU_A, oracle.GELU_C, oracle.regelu2_fwd, oracle.regelu2_bwd),
                                ("silu", oracle.SILU_A, oracle.SILU_C, oracle.resilu2_fwd, oracle.resilu2_bwd)):
        y, w = V.stepact_fwd(x, act, c, 2)
        y2, w2 = fwd(x)
        assert np.array_equal(y, y2) and np.array_equal(w, w2)
        assert np.array_equal(V.stepact_bwd(dy, w, V.family_levels(a), 2), bwd(dy, w2))
