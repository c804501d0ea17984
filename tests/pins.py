"""Independent checks ("pins") of the CPU oracle.

Each pin takes the implementation under test as an argument and returns a
non-negative error measure; the oracle must score below the stated bound, and the
planted-mistake tests feed deliberately broken variants to show that each pin
actually catches the kind of mistake it is meant to catch.

Nothing here re-derives the oracle's own formulas with the oracle's own library
calls: every pin compares against a different implementation (libm, torch), a
closed form or asymptotic series from the mathematics, a value printed in the
paper or a textbook table, brute force, or finite differences.
"""

import math
import os
from fractions import Fraction

import numpy as np
import torch
import torch.nn.functional as F

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def read_golden_constants():
    out = {}
    with open(os.path.join(GOLDEN, "constants.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            name, vals = line.split("=")
            out[name.strip()] = [float(v) for v in vals.split()]
    return out


def read_normal_cdf_table():
    xs, ps = [], []
    with open(os.path.join(GOLDEN, "normal_cdf.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            x, p = line.split()
            xs.append(float(x))
            ps.append(float(p))
    return np.array(xs), np.array(ps)


# ------------------------------------------------------------ activations

def pin_constraint(a, c):
    """|sum_i a_i c_i + (1 - a1 - a2) c3|: the constraint of eq. relus_family."""
    a1, a2 = a
    c1, c2, c3 = c
    return abs(a1 * c1 + a2 * c2 + (1.0 - a1 - a2) * c3)


def pin_gelu_table(gelu):
    """Max relative error of GELU(x)/x against the textbook Phi(x) table."""
    xs, ps = read_normal_cdf_table()
    err = 0.0
    for x, p in zip(xs, ps):
        y = float(gelu(np.array([x]))[0])
        if x == 0.0:
            err = max(err, abs(y))
        else:
            err = max(err, abs(y / x - p) / p)
    return err


def _phi_lower_tail_series(x, terms=20):
    """Phi(x) for x << 0 by the asymptotic series of Mills' ratio
    (Abramowitz & Stegun 26.2.12): Phi(x) = phi(x)/|x| * sum_k (-1)^k (2k-1)!! / x^(2k).
    The series alternates, so the truncation error is below the first omitted term."""
    t = abs(x)
    s, term = 0.0, 1.0
    for k in range(terms):
        s += term
        term *= -(2 * k + 1) / (t * t)
    dens = math.exp(-0.5 * t * t) / math.sqrt(2.0 * math.pi)
    return dens / t * s, dens / t * abs(term)


def pin_gelu_tail(gelu):
    """Max relative error of GELU against x * Phi(x) from the asymptotic series, x in [-37, -10]."""
    err = 0.0
    for x in np.linspace(-37.0, -10.0, 55):
        ref, bound = _phi_lower_tail_series(x)
        assert bound < 1e-14 * ref
        y = float(gelu(np.array([x]))[0])
        err = max(err, abs(y - x * ref) / abs(x * ref))
    return err


def pin_gelu_libm(gelu):
    """Max relative error against GELU evaluated with the C library's erfc."""
    xs = np.concatenate([np.linspace(-9.0, 9.0, 721), [-1e4, -40.0, 40.0, 1e4]])
    err = 0.0
    for x in xs:
        ref = 0.5 * x * math.erfc(-x / math.sqrt(2.0))
        y = float(gelu(np.array([x]))[0])
        if ref == 0.0:
            err = max(err, abs(y))
        else:
            err = max(err, abs(y - ref) / abs(ref))
    return err


def pin_gelu_torch(gelu):
    """Max relative error against torch's float64 erf-form GELU on [-4, 4], where
    1 + erf does not cancel badly."""
    x = np.linspace(-4.0, 4.0, 4001)
    ref = F.gelu(torch.from_numpy(x), approximate="none").numpy()
    y = gelu(x)
    mask = ref != 0
    return float(np.max(np.abs(y[mask] - ref[mask]) / np.abs(ref[mask])))


def pin_odd_part(fn, scale=1.0):
    """Max |f(x) - f(-x) - x| / max(1, |x|): GELU and SiLU both satisfy f(x) - f(-x) = x
    (Phi(x) + Phi(-x) = 1 and sigmoid(x) + sigmoid(-x) = 1)."""
    x = np.linspace(-50.0, 50.0, 2001) * scale
    d = fn(x) - fn(-x) - x
    return float(np.max(np.abs(d) / np.maximum(1.0, np.abs(x))))


def pin_silu_torch(silu):
    x = np.concatenate([np.linspace(-30.0, 30.0, 6001), [-1e4, -80.0, 80.0, 1e4]])
    ref = F.silu(torch.from_numpy(x)).numpy()
    y = silu(x)
    mask = np.abs(ref) > 1e-300
    return float(np.max(np.abs(y[mask] - ref[mask]) / np.abs(ref[mask])))


def pin_silu_direct(silu):
    """Against x / (1 + exp(-x)) with math.exp, for x where exp(-x) does not overflow."""
    err = 0.0
    for x in np.linspace(-700.0, 40.0, 1481):
        ref = x / (1.0 + math.exp(-x))
        y = float(silu(np.array([x]))[0])
        if ref != 0.0:
            err = max(err, abs(y - ref) / abs(ref))
    return err


def _kink_free_points(c, n, seed, lo=-8.0, hi=8.0, gap=1e-3):
    g = np.random.default_rng(seed)
    x = g.uniform(lo, hi, size=4 * n)
    keep = np.ones_like(x, dtype=bool)
    for ci in c:
        keep &= np.abs(x - ci) > gap
    return x[keep][:n]


def pin_levels_fd(relu_combination, derivative_levels, segment_code, a, c, seed=0):
    """Max |central FD slope of h~ - level[code]| at points at least 1e-3 from a kink."""
    x = _kink_free_points(c, 2000, seed)
    h = 1e-6
    fd = (relu_combination(x + h, a, c) - relu_combination(x - h, a, c)) / (2 * h)
    lv = derivative_levels(a)[segment_code(x, c)]
    return float(np.max(np.abs(fd - lv)))


def pin_prop43(relu_combination, a, c):
    """Prop. 4.3 / Appendix E: h~ = 0 left of every bias and h~ = x right of every bias."""
    left = np.linspace(c[0] - 50.0, c[0] - 1e-6, 200)
    right = np.linspace(c[2] + 1e-6, c[2] + 1e4, 200)
    e_left = float(np.max(np.abs(relu_combination(left, a, c))))
    e_right = float(np.max(np.abs(relu_combination(right, a, c) - right) / np.maximum(1.0, right)))
    return max(e_left, e_right)


def pin_codes_brute(segment_code, c):
    """Codes of random values against a per-element count written as a Python loop."""
    g = np.random.default_rng(1)
    x = np.concatenate([g.normal(0, 4, 500), np.array(c) + 1e-9, np.array(c) - 1e-9])
    got = segment_code(x, c)
    bad = 0
    for xi, gi in zip(x, got):
        k = 0
        for ci in c:
            if xi > ci:
                k += 1
        bad += int(k != int(gi))
    return bad


def pin_pack_layout(pack_codes, unpack_codes):
    """Hand-checked words for small code sequences plus a random round trip."""
    bad = 0
    w = pack_codes(np.array([1, 2, 3, 0], dtype=np.uint8))
    bad += int(w.size != 1 or int(w[0]) != 1 + 2 * 4 + 3 * 16)
    w = pack_codes(np.full(17, 3, dtype=np.uint8))
    bad += int(w.size != 2 or int(w[0]) != 0xFFFFFFFF or int(w[1]) != 3)
    codes = np.zeros(16, dtype=np.uint8)
    codes[15] = 2
    w = pack_codes(codes)
    bad += int(int(w[0]) != 2 << 30)
    g = np.random.default_rng(2)
    for n in (1, 15, 16, 17, 33, 1000):
        c = g.integers(0, 4, n).astype(np.uint8)
        bad += int(not np.array_equal(unpack_codes(pack_codes(c), n), c))
    return bad


def pin_bwd_fd(act_bwd, pack_codes, segment_code, relu_combination, a, c, seed=3):
    """Backward of the oracle against dy times the FD slope of h~, away from kinks."""
    x = _kink_free_points(c, 1000, seed)
    dy = np.random.default_rng(seed + 1).normal(size=x.size)
    h = 1e-6
    fd = (relu_combination(x + h, a, c) - relu_combination(x - h, a, c)) / (2 * h)
    dx = act_bwd(dy, pack_codes(segment_code(x, c)))
    return float(np.max(np.abs(dx - dy * fd)))


# ------------------------------------------------------------------ norms

def pin_ln_fwd_torch(msln_fwd, eps=1e-6, seed=0):
    g = np.random.default_rng(seed)
    x = g.normal(0.5, 2.0, size=(37, 129))
    z, rstd = msln_fwd(x, eps)
    xt = torch.from_numpy(x)
    zt = F.layer_norm(xt, (x.shape[1],), eps=eps).numpy()
    var = torch.var(xt, dim=1, unbiased=False).numpy()
    return max(float(np.max(np.abs(z - zt))),
               float(np.max(np.abs(rstd * np.sqrt(var + eps) - 1.0))))


def pin_rms_fwd_torch(msrms_fwd, eps=1e-5, seed=0):
    g = np.random.default_rng(seed)
    x = g.normal(0.5, 2.0, size=(37, 129))
    z, rstd = msrms_fwd(x, eps)
    zt = F.rms_norm(torch.from_numpy(x), (x.shape[1],), eps=eps).numpy()
    ms = np.array([sum(float(v) ** 2 for v in row) / x.shape[1] for row in x])
    return max(float(np.max(np.abs(z - zt))),
               float(np.max(np.abs(rstd * np.sqrt(ms + eps) - 1.0))))


def pin_norm_fd(fwd, bwd, eps, seed=0):
    """Backward against brute-force central differences of the forward map.

    dx_k = sum_j dz_j dz_j/dx_k, estimated by perturbing each x_k by +-h. Tiny rows."""
    g = np.random.default_rng(seed)
    worst = 0.0
    for p in (1, 2, 3, 5, 7, 16):
        x = g.normal(0.3, 1.5, size=(3, p))
        dz = g.normal(size=(3, p))
        z, rstd = fwd(x, eps)
        dx = bwd(dz, z, rstd)
        h = 1e-6
        fd = np.zeros_like(x)
        for k in range(p):
            xp = x.copy(); xp[:, k] += h
            xm = x.copy(); xm[:, k] -= h
            zp, _ = fwd(xp, eps)
            zm, _ = fwd(xm, eps)
            fd[:, k] = ((zp - zm) / (2 * h) * dz).sum(axis=1)
        scale = np.maximum(1.0, np.abs(fd))
        worst = max(worst, float(np.max(np.abs(dx - fd) / scale)))
    return worst


def pin_norm_autograd(fwd, bwd, centered, eps, seed=0):
    """Backward against torch autograd through the standard float64 norm (no affine)."""
    g = np.random.default_rng(seed)
    x = g.normal(-0.7, 3.0, size=(11, 64))
    dz = g.normal(size=x.shape)
    xt = torch.from_numpy(x).requires_grad_(True)
    if centered:
        zt = F.layer_norm(xt, (64,), eps=eps)
    else:
        zt = F.rms_norm(xt, (64,), eps=eps)
    (zt * torch.from_numpy(dz)).sum().backward()
    z, rstd = fwd(x, eps)
    dx = bwd(dz, z, rstd)
    return float(np.max(np.abs(dx - xt.grad.numpy())))


def pin_affine_merge(fwd, bwd, centered, eps, seed=0):
    """Sec. 5.2 / Appendix G: a norm with affine (alpha, beta) followed by Linear(W, b)
    equals the parameter-free norm followed by Linear(W diag(alpha), W beta + b), and
    the input gradient of the standard stack (torch autograd) equals the memory-sharing
    backward fed dz = W~^T dy. Returns the worse of the output and gradient errors."""
    g = np.random.default_rng(seed)
    rows, p, q = 9, 48, 20
    x = g.normal(0.2, 1.7, size=(rows, p))
    alpha = g.normal(1.0, 0.3, size=p)
    beta = g.normal(0.0, 0.3, size=p) if centered else np.zeros(p)
    W = g.normal(size=(q, p)) / math.sqrt(p)
    b = g.normal(size=q)
    dy = g.normal(size=(rows, q))

    xt = torch.from_numpy(x).requires_grad_(True)
    if centered:
        n = F.layer_norm(xt, (p,), weight=torch.from_numpy(alpha), bias=torch.from_numpy(beta), eps=eps)
    else:
        n = F.rms_norm(xt, (p,), weight=torch.from_numpy(alpha), eps=eps)
    y_std = n @ torch.from_numpy(W).T + torch.from_numpy(b)
    (y_std * torch.from_numpy(dy)).sum().backward()

    W_m = W * alpha[None, :]
    b_m = W @ beta + b
    z, rstd = fwd(x, eps)
    y_ms = z @ W_m.T + b_m
    dx = bwd(dy @ W_m, z, rstd)
    return max(float(np.max(np.abs(y_ms - y_std.detach().numpy()))),
               float(np.max(np.abs(dx - xt.grad.numpy()))))


def pin_norm_invariants(fwd, bwd, centered, eps, seed=0):
    """Identities of the exact maps, for rows of width 257:
    LN: sum z = 0 and sum dx = 0; both: |z|^2 = p (1 - eps rstd^2) and
    z^T dx = eps rstd^3 z^T dz; LN with dz constant along the row gives dx = 0."""
    g = np.random.default_rng(seed)
    p = 257
    x = g.normal(1.0, 0.05, size=(16, p))  # small spread so eps matters
    dz = g.normal(size=x.shape)
    z, rstd = fwd(x, eps)
    dx = bwd(dz, z, rstd)
    errs = [np.abs((z * z).sum(1) - p * (1 - eps * rstd ** 2)) / p,
            np.abs((z * dx).sum(1) - eps * rstd ** 3 * (z * dz).sum(1)) / np.maximum(1.0, rstd)]
    if centered:
        errs.append(np.abs(z.sum(1)))
        errs.append(np.abs(dx.sum(1)) / np.maximum(1.0, rstd))
        dconst = bwd(np.ones_like(dz) * 2.5, z, rstd)
        errs.append(np.abs(dconst).max(1) / np.maximum(1.0, rstd))
    return float(max(np.max(e) for e in errs))


# ----------------------------------------------------------------- dtypes

def _exact_bf16_round(v):
    """Nearest bf16 value (ties to even) by exact rational search over the two
    bf16 neighbours that bracket v."""
    fv = Fraction(v)
    if fv == 0:
        return 0.0
    sign = -1 if fv < 0 else 1
    av = abs(fv)
    e = 0
    while Fraction(2) ** e > av:
        e -= 1
    while Fraction(2) ** (e + 1) <= av:
        e += 1
    e = max(e, -126)
    ulp = Fraction(2) ** (e - 7)
    k = av // ulp
    lo, hi = k * ulp, (k + 1) * ulp
    dlo, dhi = av - lo, hi - av
    if dlo < dhi or (dlo == dhi and k % 2 == 0):
        r = lo
    else:
        r = hi
    return sign * float(r)


def pin_bf16_rounding(round_to_dtype, seed=0):
    """Count of values whose bf16 rounding differs from exact rational rounding,
    over random values, exact ties, ties +- one fp64 ulp and subnormal-range values."""
    g = np.random.default_rng(seed)
    vals = list(g.normal(0, 10, 300)) + list(g.normal(0, 1e-38, 50))
    for m in range(128, 256, 7):               # exact midpoints between bf16 values
        mid = (m + 0.5) * 2.0 ** -7
        vals += [mid, -mid, math.nextafter(mid, 0), math.nextafter(mid, 2)]
    vals += [2.0 ** -133 * 0.5, 2.0 ** -133 * 1.5, 1e-40, 3.0, 1e4, -1e4]
    got = round_to_dtype(np.array(vals), "bf16")
    return sum(int(_exact_bf16_round(v) != float(r)) for v, r in zip(vals, got))


# ----------------------------------------------------------------- SwiGLU

def pin_swiglu_fd(fwd, bwd, relu_combination, a, c, seed=5):
    """Backward of h = SiLU(g) * u under Approx-BP against finite differences of the
    approximate network h~(g) * u for dg (away from kinks) and of the exact product
    in u for du (where du/du of s * u is s). Returns the worse absolute error."""
    g = _kink_free_points(c, 800, seed)
    r = np.random.default_rng(seed + 1)
    u = r.normal(size=g.size)
    dh = r.normal(size=g.size)
    h, s, words = fwd(g, u)
    dg, du = bwd(dh, u, s, words)
    eps = 1e-6
    fd_g = (relu_combination(g + eps, a, c) * u - relu_combination(g - eps, a, c) * u) / (2 * eps)
    s_ref = F.silu(torch.from_numpy(g)).numpy()                   # SiLU from another library
    fd_u = (s_ref * (u + eps) - s_ref * (u - eps)) / (2 * eps)
    return max(float(np.max(np.abs(dg - dh * fd_g))), float(np.max(np.abs(du - dh * fd_u))))


def pin_swiglu_reduces_to_resilu2(fwd, bwd, act_fwd, act_bwd, seed=6):
    """With u = 1 the fused op is ReSiLU2 itself: h = s = SiLU(g), same codes, dg = ReSiLU2's dx."""
    g = np.random.default_rng(seed).normal(0, 3, size=777)
    one = np.ones_like(g)
    dh = np.random.default_rng(seed + 1).normal(size=g.size)
    h, s, words = fwd(g, one)
    y, w2 = act_fwd(g)
    dg, du = bwd(dh, one, s, words)
    bad = int(not np.array_equal(words, w2))
    err = max(float(np.max(np.abs(h - y))), float(np.max(np.abs(s - y))),
              float(np.max(np.abs(dg - act_bwd(dh, w2)))), float(np.max(np.abs(du - dh * y))))
    return bad + err


# ------------------------------------------------- general k-bit family

def pin_stepact_fd(stepact_fwd, stepact_bwd, relu_family, a, c, bits, act, seed=11):
    """Composed k-bit forward + backward against what the mathematics fixes, at points
    at least 1e-3 from every bias:
    * the forward value against torch's float64 GELU (erf form, on [-4, 4]) or SiLU;
    * dx of the backward, fed the forward's packed words, against dy times the central
      finite-difference slope of the ReLU combination h~_{a,c} (eq. relus_family for
      general k; the slope of segment j is the sum of the first j weights).
    Returns the larger of the two maximum errors (relative for the value, absolute for
    dx with dy ~ N(0, 1))."""
    x = _kink_free_points(c, 1500, seed, lo=min(c) - 3.0, hi=max(c) + 3.0)
    # odd-length tail so that the last packed word is partial
    x = x[: x.size - (x.size % (32 // bits)) - 1]
    dy = np.random.default_rng(seed + 1).normal(size=x.size)
    y, words = stepact_fwd(x, act, c, bits)
    xt = torch.from_numpy(x)
    ref = (F.gelu(xt, approximate="none") if act == "gelu" else F.silu(xt)).numpy()
    # torch's erf-form GELU cancels for x < -4 (1 + erf), so the value is compared on
    # [-4, 4] for GELU, everywhere for SiLU
    mask = (ref != 0) & ((np.abs(x) <= 4.0) if act == "gelu" else True)
    e_y = float(np.max(np.abs(y[mask] - ref[mask]) / np.abs(ref[mask])))
    # levels as the slopes of the combination itself, not through the oracle's helper;
    # h~ is linear within 1e-3 of every point used, so a step of 1e-4 is exact up to
    # rounding
    h = 1e-4
    fd = (relu_family(x + h, a, c) - relu_family(x - h, a, c)) / (2 * h)
    seg_slopes = np.zeros(len(c) + 1)
    for j in range(len(c) + 1):
        lo = c[j - 1] if j > 0 else c[0] - 10.0
        hi = c[j] if j < len(c) else c[-1] + 10.0
        mid = 0.5 * (lo + hi)
        seg_slopes[j] = (relu_family(np.array([mid + h]), a, c)[0]
                         - relu_family(np.array([mid - h]), a, c)[0]) / (2 * h)
    dx = stepact_bwd(dy, words, seg_slopes, bits)
    e_dx = float(np.max(np.abs(dx - dy * fd)))
    return max(e_y, e_dx)


def pin_stepact_words_brute(stepact_fwd, c, bits, act="gelu", seed=12):
    """Packed words of the composed forward against codes counted per element in a
    Python loop and packed bit by bit (floor(32/k) codes per word, least significant
    first, zero tail). Returns the number of words that differ (or -1 on a size
    mismatch)."""
    per = 32 // bits
    r = np.random.default_rng(seed)
    x = np.concatenate([r.normal(0, 3, 3 * per + 5), np.asarray(c) + 1e-9, np.asarray(c) - 1e-9])
    _, words = stepact_fwd(x, act, c, bits)
    want = [0] * ((x.size + per - 1) // per)
    for i, xi in enumerate(x):
        k = 0
        for ci in c:
            if xi > ci:
                k += 1
        want[i // per] |= k << (bits * (i % per))
    if len(words) != len(want):
        return -1
    return sum(int(int(w) != v) for w, v in zip(words, want))
