"""The offline constant search (App. E objective; App. I derivative objective)."""

import math

import numpy as np
import pytest
from scipy import integrate
from scipy.stats import norm

import oracle
from oracle import variants as OV
from paper_2406_16282_amd import fit


def quad_objective(f, a, c, B):
    pts = sorted(set([-B, B] + [float(v) for v in c if -B < v < B]))
    total = 0.0
    for lo, hi in zip(pts[:-1], pts[1:]):
        total += integrate.quad(lambda x: f(x, a, c) ** 2, lo, hi, epsabs=1e-14, epsrel=1e-12, limit=200)[0]
    return total


def test_tail_bounds_of_appendix_e():
    assert fit.domain("gelu") == pytest.approx(math.sqrt(-2 * math.log(1e-8)), rel=1e-15)
    assert fit.domain("gelu") == pytest.approx(6.0697, abs=1e-4)
    assert fit.domain("silu") == pytest.approx(38.2277, abs=1e-4)


@pytest.mark.parametrize("act", ["gelu", "silu"])
def test_function_objective_against_quadrature(act):
    a, c = (oracle.GELU_A, oracle.GELU_C) if act == "gelu" else (oracle.SILU_A, oracle.SILU_C)
    hfun = oracle.gelu if act == "gelu" else oracle.silu
    f = lambda x, a_, c_: float(hfun(np.array([x]))[0] - oracle.relu_combination(np.array([x]), a_, c_)[0])
    ref = quad_objective(f, a, c, fit.domain(act))
    assert fit.objective(act, a, c) == pytest.approx(ref, rel=1e-9)


def test_derivative_objective_against_quadrature():
    a, c = OV.REGELU2D_A, OV.REGELU2D_C
    d = lambda x: norm.cdf(x) + x * norm.pdf(x)
    f = lambda x, a_, c_: d(x) - OV.family_levels(a_)[int(OV.family_code(np.array([x]), c_)[0])]
    ref = quad_objective(f, a, c, fit.domain("gelu"))
    assert fit.objective("gelu", a, c, "derivative") == pytest.approx(ref, rel=1e-8)


@pytest.mark.parametrize("act,kind", [("gelu", "function"), ("silu", "function"), ("gelu", "derivative")])
def test_refit_reaches_the_printed_constants(act, kind):
    if kind == "derivative":
        a0, c0 = OV.REGELU2D_A, OV.REGELU2D_C
    else:
        a0, c0 = (oracle.GELU_A, oracle.GELU_C) if act == "gelu" else (oracle.SILU_A, oracle.SILU_C)
    a, c, val = fit.fit(act, 2, kind, starts=4)
    assert val <= fit.objective(act, a0, c0, kind) * (1 + 1e-9)
    assert np.allclose(a, a0, atol=2e-3)
    assert np.allclose(c, c0, atol=3e-2 * max(1.0, abs(c0[0]) / 3))


def test_more_bits_fit_closer():
    _, _, v1 = fit.fit("gelu", 1, starts=2)
    _, _, v2 = fit.fit("gelu", 2, starts=2)
    _, _, v4 = fit.fit("gelu", 4, starts=1)
    assert v1 > v2 > 10 * v4
