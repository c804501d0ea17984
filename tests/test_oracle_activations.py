"""Pins of the oracle's ReGELU2 / ReSiLU2 (Sec. 4.2, eq. relus_family, Prop. 4.3, Appendix E)."""

import math

import numpy as np
import pytest

import oracle
import pins

ACTS = {
    "gelu": (oracle.GELU_A, oracle.GELU_C, oracle.regelu2_bwd),
    "silu": (oracle.SILU_A, oracle.SILU_C, oracle.resilu2_bwd),
}


def test_constants_match_appendix_e():
    g = pins.read_golden_constants()
    assert list(oracle.GELU_A) == g["gelu_a"]
    assert list(oracle.GELU_C) == g["gelu_c"]
    assert list(oracle.SILU_A) == g["silu_a"]
    assert list(oracle.SILU_C) == g["silu_c"]


def test_main_text_values_are_roundings_of_appendix_values():
    g = pins.read_golden_constants()
    for name in ("gelu_a", "gelu_c", "silu_a", "silu_c"):
        for full, short in zip(g[name], g[name + "_short"]):
            digits = 4 - int(math.floor(math.log10(abs(full))))
            assert round(full, digits - 1) == pytest.approx(short, rel=0, abs=0.6 * 10 ** -(digits - 1))


@pytest.mark.parametrize("act", ["gelu", "silu"])
def test_constraint_of_relu_combination(act):
    a, c, _ = ACTS[act]
    assert pins.pin_constraint(a, c) < 1e-14


def test_gelu_textbook_table():
    assert pins.pin_gelu_table(oracle.gelu) < 1e-14


def test_gelu_lower_tail_asymptotic_series():
    assert pins.pin_gelu_tail(oracle.gelu) < 1e-12


def test_gelu_against_libm_erfc():
    assert pins.pin_gelu_libm(oracle.gelu) < 1e-13


def test_gelu_against_torch():
    assert pins.pin_gelu_torch(oracle.gelu) < 1e-11


@pytest.mark.parametrize("fn", [oracle.gelu, oracle.silu])
def test_odd_part_identity(fn):
    assert pins.pin_odd_part(fn) < 1e-14


def test_silu_against_torch_and_direct_formula():
    assert pins.pin_silu_torch(oracle.silu) < 1e-14
    assert pins.pin_silu_direct(oracle.silu) < 1e-14


@pytest.mark.parametrize("act", ["gelu", "silu"])
def test_levels_are_slopes_of_relu_combination(act):
    a, c, _ = ACTS[act]
    assert pins.pin_levels_fd(oracle.relu_combination, oracle.derivative_levels,
                              oracle.segment_code, a, c) < 1e-8


@pytest.mark.parametrize("act", ["gelu", "silu"])
def test_prop_4_3_limits(act):
    a, c, _ = ACTS[act]
    assert pins.pin_prop43(oracle.relu_combination, a, c) < 1e-12
    # h - h~ -> 0 at both ends (Prop. 4.3, item 1)
    h = oracle.gelu if act == "gelu" else oracle.silu
    for x in (-1e4, 1e4):
        assert abs(h(np.array([x]))[0] - oracle.relu_combination(np.array([x]), a, c)[0]) < 1e-9


@pytest.mark.parametrize("act", ["gelu", "silu"])
def test_codes_brute_force(act):
    _, c, _ = ACTS[act]
    assert pins.pin_codes_brute(oracle.segment_code, c) == 0


def test_codes_worked_bf16_values():
    # Hand-checkable against the printed biases c = (-3.18588..., -0.00117882..., 3.19083...):
    # every value below is exactly representable in bf16.
    cases = [(-3.1875, 0), (-3.171875, 1), (-0.00118255615234375, 1),
             (-0.0011749267578125, 2), (0.0, 2), (-0.0, 2), (3.1875, 2), (3.203125, 3)]
    for x, want in cases:
        assert int(oracle.segment_code(np.array([x]), oracle.GELU_C)[0]) == want, x


@pytest.mark.parametrize("act", ["gelu", "silu"])
def test_code_flips_between_fp32_neighbours_of_each_bias(act):
    _, c, _ = ACTS[act]
    for i, ci in enumerate(c):
        f = np.float32(ci)
        assert float(f) != ci, "bias representable in fp32: tie rule would matter"
        lo = f if float(f) < ci else np.nextafter(f, np.float32(-np.inf))
        hi = np.nextafter(lo, np.float32(np.inf))
        assert float(lo) < ci < float(hi)
        codes = oracle.segment_code(np.array([lo, hi], dtype=np.float64), c)
        assert list(codes) == [i, i + 1]


def test_pack_layout():
    assert pins.pin_pack_layout(oracle.pack_codes, oracle.unpack_codes) == 0


def test_pack_tail_bits_zero_and_word_count():
    for n in (1, 7, 16, 17, 31, 32, 33):
        w = oracle.pack_codes(np.full(n, 3, dtype=np.uint8))
        assert w.size == oracle.codes_words(n) == (n + 15) // 16
        rem = n % 16
        if rem:
            assert int(w[-1]) == (1 << (2 * rem)) - 1


@pytest.mark.parametrize("act", ["gelu", "silu"])
def test_backward_is_dy_times_fd_slope(act):
    a, c, bwd = ACTS[act]
    assert pins.pin_bwd_fd(bwd, oracle.pack_codes, oracle.segment_code,
                           oracle.relu_combination, a, c) < 1e-7


def test_level_values():
    lg = oracle.derivative_levels(oracle.GELU_A)
    ls = oracle.derivative_levels(oracle.SILU_A)
    assert lg[0] == 0.0 and lg[3] == 1.0 and ls[0] == 0.0 and ls[3] == 1.0
    assert lg[2] == pytest.approx(1.0487405950855513, rel=1e-15)
    assert ls[2] == pytest.approx(1.0403218566243821, rel=1e-15)


def test_fwd_bwd_shapes_and_finite_guard():
    x = np.linspace(-5, 5, 37).reshape(1, 37)
    y, w = oracle.regelu2_fwd(x)
    assert y.shape == x.shape and w.size == 3
    dx = oracle.regelu2_bwd(np.ones_like(x), w)
    assert dx.shape == x.shape
    with pytest.raises(ValueError):
        oracle.resilu2_fwd(np.array([np.inf]))
