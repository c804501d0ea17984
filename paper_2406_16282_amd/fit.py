"""Offline search for the weights and biases of a ReLU combination (Sec. 4.2, App. E/I).

For an activation h (GELU or SiLU) and k bits, find a (2^k - 2 free weights; the last
weight is 1 - sum a) and increasing biases c (2^k - 1 of them) minimising

    "function"   : integral over [-B, B] of (h(x) - h~_{a,c}(x))^2 dx       (eq. objective)
    "derivative" : integral over [-B, B] of (h'(x) - h~'_{a,c}(x))^2 dx     (Appendix I)

where the tails beyond B are negligible: B = sqrt(-2 ln eps) for GELU and
B = -2 ln(eps / 2) for SiLU with eps = 1e-8 (Appendix E's tail bounds). The integral
is evaluated with Gauss-Legendre panels whose edges include every bias (h~ is
piecewise linear, so each panel integrand is smooth). Biases are parameterised by the
first one and log-gaps, which keeps them ordered. The search is multi-start local
optimisation (L-BFGS-B), optionally seeded by scipy's dual annealing (a generalised
simulated annealing, the paper's search method).

The printed constants of Appendix E are the contract for ReGELU2/ReSiLU2; this tool
regenerates such tables for other k (fed to ``stepact_fwd``/``stepact_bwd``) and
checks the printed ones.

Command line: python -m paper_2406_16282_amd.fit --act gelu --bits 2
"""

import argparse
import math

import numpy as np
from scipy import optimize, special

EPS_TAIL = 1e-8


def domain(act):
    """Half-width B of the integration interval (Appendix E)."""
    if act == "gelu":
        return math.sqrt(-2.0 * math.log(EPS_TAIL))
    if act == "silu":
        return -2.0 * math.log(EPS_TAIL / 2.0)
    raise ValueError("act must be 'gelu' or 'silu'")


def h(act, x):
    if act == "gelu":
        return 0.5 * x * special.erfc(-x / math.sqrt(2.0))
    return x * special.expit(x)


def dh(act, x):
    if act == "gelu":
        return special.ndtr(x) + x * np.exp(-0.5 * x * x) / math.sqrt(2.0 * math.pi)
    s = special.expit(x)
    return s + x * s * (1.0 - s)


def _weights(a):
    a = np.asarray(a, dtype=np.float64)
    return np.append(a, 1.0 - a.sum())


def relu_comb(x, a, c):
    w = _weights(a)
    return sum(wi * np.maximum(x - ci, 0.0) for wi, ci in zip(w, c))


def relu_comb_slope(x, a, c):
    w = _weights(a)
    return sum(wi * (x > ci) for wi, ci in zip(w, c))


_GL_X, _GL_W = np.polynomial.legendre.leggauss(48)


def _panels(c, B, width=0.5):
    edges = np.unique(np.clip(np.concatenate([[-B, B], np.asarray(c, dtype=np.float64)]), -B, B))
    out = []
    for lo, hi in zip(edges[:-1], edges[1:]):
        m = max(1, int(math.ceil((hi - lo) / width)))
        e = np.linspace(lo, hi, m + 1)
        out.extend(zip(e[:-1], e[1:]))
    return np.array(out)


def objective(act, a, c, kind="function"):
    """The L2 objective for the combination (a, c)."""
    B = domain(act)
    p = _panels(c, B)
    mid = 0.5 * (p[:, 0] + p[:, 1])[:, None]
    half = 0.5 * (p[:, 1] - p[:, 0])[:, None]
    x = mid + half * _GL_X[None, :]
    if kind == "function":
        r = h(act, x) - relu_comb(x, a, c)
    elif kind == "derivative":
        r = dh(act, x) - relu_comb_slope(x, a, c)
    else:
        raise ValueError("kind must be 'function' or 'derivative'")
    return float(np.sum(half * _GL_W[None, :] * r * r))


def _unpack(theta, m):
    a = theta[: m - 1]
    c0 = theta[m - 1]
    gaps = np.exp(theta[m:])
    c = c0 + np.concatenate([[0.0], np.cumsum(gaps)])
    return a, c


def _pack(a, c):
    c = np.asarray(c, dtype=np.float64)
    return np.concatenate([np.asarray(a, dtype=np.float64), [c[0]], np.log(np.diff(c))])


def fit(act, bits=2, kind="function", starts=8, seed=0, anneal=False, x0=None):
    """Return (a, c, objective) of the best local optimum over the starts."""
    m = (1 << bits) - 1
    B = domain(act)
    rng = np.random.default_rng(seed)
    f = lambda th: objective(act, *_unpack(th, m), kind=kind)
    inits = []
    if x0 is not None:
        inits.append(_pack(*x0))
    if anneal:
        lo = np.concatenate([-2.0 * np.ones(m - 1), [-B / 2], np.full(m - 1, math.log(1e-3))])
        hi = np.concatenate([2.0 * np.ones(m - 1), [0.0], np.full(m - 1, math.log(B))])
        res = optimize.dual_annealing(f, list(zip(lo, hi)), seed=seed, maxiter=200)
        inits.append(res.x)
    span = min(B, 8.0)
    while len(inits) < starts:
        c = np.sort(rng.uniform(-span / 2, span / 2, m))
        c = c + np.arange(m) * 1e-3
        a = rng.normal(0.0, 0.5, m - 1)
        inits.append(_pack(a, c))
    best = None
    for th in inits:
        r = optimize.minimize(f, th, method="L-BFGS-B", options={"maxiter": 2000, "ftol": 1e-15, "gtol": 1e-12})
        if best is None or r.fun < best.fun:
            best = r
    a, c = _unpack(best.x, m)
    return a, c, float(best.fun)


def main():
    ap = argparse.ArgumentParser(description="Fit a ReLU combination to GELU or SiLU")
    ap.add_argument("--act", choices=("gelu", "silu"), default="gelu")
    ap.add_argument("--bits", type=int, choices=(1, 2, 3, 4), default=2)
    ap.add_argument("--objective", choices=("function", "derivative"), default="function")
    ap.add_argument("--starts", type=int, default=8)
    ap.add_argument("--anneal", action="store_true", help="seed the search with dual annealing")
    ap.add_argument("--seed", type=int, default=0)
    args = ap.parse_args()
    a, c, val = fit(args.act, args.bits, args.objective, args.starts, args.seed, args.anneal)
    levels = np.concatenate([[0.0], np.cumsum(a), [1.0]])
    print(f"a = {list(map(float, a))}")
    print(f"c = {list(map(float, c))}")
    print(f"levels = {list(map(float, levels))}")
    print(f"objective = {val:.10g}")


if __name__ == "__main__":
    main()
