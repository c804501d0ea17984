"""Property tests of the oracle (hypothesis, fixed seed)."""

import numpy as np
from hypothesis import given, settings, strategies as st

import oracle
import pins

SETTINGS = settings(max_examples=200, deadline=None, derandomize=True)


@SETTINGS
@given(st.lists(st.integers(0, 3), min_size=0, max_size=100))
def test_pack_round_trip(codes):
    c = np.array(codes, dtype=np.uint8)
    w = oracle.pack_codes(c)
    assert w.size == (len(codes) + 15) // 16
    assert np.array_equal(oracle.unpack_codes(w, len(codes)), c)


@SETTINGS
@given(st.floats(-1e4, 1e4, allow_nan=False), st.floats(-1e4, 1e4, allow_nan=False))
def test_codes_monotone(a, b):
    lo, hi = min(a, b), max(a, b)
    for c in (oracle.GELU_C, oracle.SILU_C):
        assert oracle.segment_code(np.array([lo]), c)[0] <= oracle.segment_code(np.array([hi]), c)[0]


@SETTINGS
@given(st.floats(-3e38, 3e38, allow_nan=False, allow_infinity=False))
def test_bf16_rounding_is_nearest_even(v):
    r = float(oracle.round_to_dtype(np.array([v]), "bf16")[0])
    assert r == pins._exact_bf16_round(v)
