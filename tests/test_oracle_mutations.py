"""Planted mistakes: each pin must reject a plausible error in the oracle.

Every mutant below is a broken copy of one oracle step (a dropped term, a wrong
sign or index, a transposed layout, a typo in a constant). The test passes only if
the pin that guards that step scores the mutant above the bound the real oracle
meets, so a pin that cannot see the mistake fails here. Mistakes are planted in
local CPU functions only.
"""

import math

import numpy as np
from scipy.special import erfc

import oracle
from oracle import norms as onorms
import pins


def test_gelu_sign_error_caught():
    bad = lambda x: 0.5 * np.asarray(x) * erfc(np.asarray(x) / math.sqrt(2.0))
    assert pins.pin_gelu_table(bad) > 1e-3


def test_gelu_tanh_approximation_caught():
    def tanh_gelu(x):
        x = np.asarray(x, dtype=np.float64)
        return 0.5 * x * (1 + np.tanh(math.sqrt(2 / math.pi) * (x + 0.044715 * x ** 3)))
    assert pins.pin_gelu_table(tanh_gelu) > 1e-6 or pins.pin_gelu_libm(tanh_gelu) > 1e-6


def test_gelu_one_plus_erf_cancellation_caught():
    from scipy.special import erf
    naive = lambda x: 0.5 * np.asarray(x) * (1 + erf(np.asarray(x) / math.sqrt(2.0)))
    assert pins.pin_gelu_tail(naive) > 1e-3


def test_silu_wrong_sign_caught():
    bad = lambda x: np.asarray(x) / (1 + np.exp(np.asarray(x, dtype=np.float64)))
    with np.errstate(over="ignore"):
        assert pins.pin_silu_torch(bad) > 1e-3


def test_constant_typo_caught():
    a = list(oracle.GELU_A)
    c = list(oracle.GELU_C)
    c[2] = 3.190842613414926          # one digit changed
    assert pins.pin_constraint(a, c) > 1e-10
    a = list(oracle.SILU_A)
    a[1] = 1.080925428529686          # two digits swapped
    assert pins.pin_constraint(a, oracle.SILU_C) > 1e-14


def test_non_cumulative_levels_caught():
    bad_levels = lambda a: np.array([0.0, a[0], a[1], 1.0])
    assert pins.pin_levels_fd(oracle.relu_combination, bad_levels, oracle.segment_code,
                              oracle.GELU_A, oracle.GELU_C) > 1e-2


def test_reversed_codes_caught():
    bad_code = lambda x, c: 3 - oracle.segment_code(x, c)
    assert pins.pin_levels_fd(oracle.relu_combination, oracle.derivative_levels, bad_code,
                              oracle.SILU_A, oracle.SILU_C) > 1e-2
    assert pins.pin_codes_brute(bad_code, oracle.SILU_C) > 0


def test_msb_first_packing_caught():
    def pack_msb(codes):
        codes = np.asarray(codes).reshape(-1)
        words = np.zeros((codes.size + 15) // 16, dtype=np.uint32)
        for slot in range(16):
            part = codes[slot::16].astype(np.uint32)
            words[: part.size] |= part << np.uint32(30 - 2 * slot)
        return words
    def unpack_msb(words, n):
        out = np.empty(words.size * 16, dtype=np.uint8)
        for slot in range(16):
            out[slot::16] = (words >> np.uint32(30 - 2 * slot)) & np.uint32(3)
        return out[:n]
    assert pins.pin_pack_layout(pack_msb, unpack_msb) > 0


def test_backward_level_index_off_by_one_caught():
    def bad_bwd(dy, words):
        codes = oracle.unpack_codes(words, np.asarray(dy).size)
        lv = oracle.derivative_levels(oracle.GELU_A)
        return np.asarray(dy) * lv[np.minimum(codes + 1, 3)]
    assert pins.pin_bwd_fd(bad_bwd, oracle.pack_codes, oracle.segment_code,
                           oracle.relu_combination, oracle.GELU_A, oracle.GELU_C) > 1e-2


def _ln_bwd_without_mean(dz, z, rstd):
    return onorms._bwd(dz, z, rstd, centered=False)


def _ln_bwd_sign_flip(dz, z, rstd):
    dz = np.asarray(dz); z = np.asarray(z); p = z.shape[1]
    h_dz = dz - dz.mean(axis=1, keepdims=True)
    return rstd[:, None] * (h_dz + z * ((z * dz).sum(1, keepdims=True) / p))


def _rms_bwd_double_mean(dz, z, rstd):
    dz = np.asarray(dz); z = np.asarray(z); p = z.shape[1]
    return rstd[:, None] * (dz - z * ((z * dz).sum(1, keepdims=True) / p / p))


def _ln_fwd_eps_outside(x, eps):
    x = np.asarray(x, dtype=np.float64); p = x.shape[1]
    hx = x - x.mean(1, keepdims=True)
    sigma = np.sqrt((hx * hx).sum(1) / p) + eps
    return hx / sigma[:, None], 1 / sigma


def _ln_fwd_unbiased(x, eps):
    x = np.asarray(x, dtype=np.float64); p = x.shape[1]
    hx = x - x.mean(1, keepdims=True)
    sigma = np.sqrt((hx * hx).sum(1) / (p - 1) + eps)
    return hx / sigma[:, None], 1 / sigma


def test_ln_backward_dropped_mean_term_caught():
    assert pins.pin_norm_fd(oracle.msln_fwd, _ln_bwd_without_mean, 1e-6) > 1e-3


def test_ln_backward_sign_flip_caught():
    assert pins.pin_norm_fd(oracle.msln_fwd, _ln_bwd_sign_flip, 1e-6) > 1e-3
    assert pins.pin_norm_autograd(oracle.msln_fwd, _ln_bwd_sign_flip, True, 1e-5) > 1e-3


def test_rms_backward_wrong_scale_caught():
    assert pins.pin_norm_fd(oracle.msrms_fwd, _rms_bwd_double_mean, 1e-5) > 1e-3


def test_ln_forward_eps_outside_sqrt_caught():
    assert pins.pin_ln_fwd_torch(_ln_fwd_eps_outside, eps=1e-2) > 1e-4


def test_ln_forward_unbiased_variance_caught():
    assert pins.pin_ln_fwd_torch(_ln_fwd_unbiased) > 1e-4


def test_rms_forward_with_centering_caught():
    assert pins.pin_rms_fwd_torch(oracle.msln_fwd) > 1e-3


def test_bwd_using_input_instead_of_output_caught():
    # A backward that treats the saved tensor as the un-normalised input breaks the
    # affine-merge equivalence.
    def fwd_returning_x(x, eps):
        z, rstd = oracle.msln_fwd(x, eps)
        return np.asarray(x, dtype=np.float64), rstd
    assert pins.pin_affine_merge(fwd_returning_x, oracle.msln_bwd, True, 1e-6) > 1e-3


def test_bf16_truncation_caught():
    def trunc(x, dtype):
        x = np.asarray(x, dtype=np.float64).astype(np.float32)
        return ((x.view(np.uint32) & np.uint32(0xFFFF0000)).view(np.float32)).astype(np.float64)
    assert pins.pin_bf16_rounding(trunc) > 0


def test_swiglu_du_from_codes_instead_of_s_caught():
    def bad_bwd(dh, u, s, words):
        dg, du = oracle.reswiglu2_bwd(dh, u, s, words)
        return dg, dh * u   # product rule with the wrong factor
    assert pins.pin_swiglu_fd(oracle.reswiglu2_fwd, bad_bwd, oracle.relu_combination,
                              oracle.SILU_A, oracle.SILU_C) > 1e-2


def test_swiglu_dg_without_u_caught():
    def bad_bwd(dh, u, s, words):
        dg, du = oracle.reswiglu2_bwd(dh, np.ones_like(u), s, words)
        return dg, dh * s
    assert pins.pin_swiglu_fd(oracle.reswiglu2_fwd, bad_bwd, oracle.relu_combination,
                              oracle.SILU_A, oracle.SILU_C) > 1e-2


# ------------------------------------------------- general k-bit family

def _kbit_table(bits):
    r = np.random.default_rng(200 + bits)
    m = (1 << bits) - 1
    return list(r.normal(0, 0.5, m - 1)), list(np.linspace(-3.0, 3.0, m))


def test_stepact_unpack_with_wrong_width_caught():
    from oracle import variants as V
    for bits, wrong in ((3, 2), (2, 4), (4, 3), (1, 2)):
        def bad_bwd(dy, words, levels, b, _w=wrong):
            dy = np.asarray(dy, dtype=np.float64)
            codes = V.unpack_bits(words, _w, dy.size) % len(levels)
            return dy * np.asarray(levels)[codes]
        a, c = _kbit_table(bits)
        try:
            err = pins.pin_stepact_fd(V.stepact_fwd, bad_bwd, V.relu_family, a, c, bits, "gelu")
        except ValueError:
            continue   # a wider field yields too few codes: the shape mismatch is loud
        assert err > 1e-2


def test_stepact_level_index_off_by_one_caught():
    from oracle import variants as V
    for bits in (1, 2, 3, 4):
        def bad_bwd(dy, words, levels, b):
            dy = np.asarray(dy, dtype=np.float64)
            codes = V.unpack_bits(words, b, dy.size)
            return dy * np.asarray(levels)[np.minimum(codes + 1, len(levels) - 1)]
        a, c = _kbit_table(bits)
        assert pins.pin_stepact_fd(V.stepact_fwd, bad_bwd, V.relu_family, a, c, bits, "silu") > 1e-2


def test_stepact_wrong_activation_or_packing_caught():
    from oracle import variants as V
    def swapped_act(x, act, c, bits):
        return V.stepact_fwd(x, "silu" if act == "gelu" else "gelu", c, bits)
    a, c = _kbit_table(3)
    assert pins.pin_stepact_fd(swapped_act, V.stepact_bwd, V.relu_family, a, c, 3, "gelu") > 1e-3
    def packed_as_k2(x, act, c, bits):
        y, _ = V.stepact_fwd(x, act, c, bits)
        return y, V.pack_bits(np.minimum(V.family_code(x, c), 3), 2)
    assert pins.pin_stepact_words_brute(packed_as_k2, c, 3) != 0
    def msb_first(x, act, c, bits):
        y, _ = V.stepact_fwd(x, act, c, bits)
        codes = V.family_code(x, c)
        per = 32 // bits
        w = np.zeros(V.words_for(bits, codes.size), dtype=np.uint32)
        for slot in range(per):
            part = codes[slot::per].astype(np.uint32)
            w[: part.size] |= part << np.uint32(bits * (per - 1 - slot))
        return y, w
    assert pins.pin_stepact_words_brute(msb_first, c, 3) != 0
