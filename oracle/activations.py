"""ReGELU2 and ReSiLU2 in float64 (Sec. 4.2 and Appendix E).

Test infrastructure only (see the package docstring).

The method keeps the exact activation in the forward pass and replaces its
derivative in the backward pass by the derivative of a combination of three
ReLUs (eq. relus_family with k = 2):

    h~(x) = a1 ReLU(x - c1) + a2 ReLU(x - c2) + (1 - a1 - a2) ReLU(x - c3).

Its derivative is a step function with four segments (Prop. 4.3, item 2), so the
backward pass only needs to know which segment each input fell in: a 2-bit code.

Readings where the paper leaves a choice open:

* Code of x = number of biases c_i strictly below x. Equality cannot occur for
  fp32 or bf16 inputs because none of the six biases is representable in either
  format; strict ">" matches ReLU'(0) = 0.
* Derivative on segment j = sum of the first j ReLU weights, i.e.
  [0, a1, a1 + a2, 1]; the last level is exactly 1 because the weights sum to 1
  (h~(x) = x to the right of every bias, Appendix E).
* Packing: code of flat element i is stored in bits [2(i mod 16), 2(i mod 16)+1]
  of 32-bit word floor(i/16), least significant bits first, unused tail bits 0.
  The paper only fixes "2 bits per element"; the layout is this implementation's.
"""

import math

import numpy as np
from scipy.special import erfc, expit

# Appendix E: quasi-optimal weights a* and biases c* found by simulated annealing
# ("adopted in our code"); Sec. 4.2 prints the same values rounded to 4-5 digits.
GELU_A = (-0.04922261145617846, 1.0979632065417297)
GELU_C = (-3.1858810036855245, -0.001178821281161997, 3.190832613414926)
SILU_A = (-0.04060357190528599, 1.080925428529668)
SILU_C = (-6.3050461001646445, -0.0008684942046214787, 6.325815242089708)


def relu_combination(x, a, c):
    """h~_{a,c}(x) of eq. relus_family for k = 2 (three ReLUs, last weight 1 - a1 - a2)."""
    x = np.asarray(x, dtype=np.float64)
    a1, a2 = a
    c1, c2, c3 = c
    relu = lambda v: np.maximum(v, 0.0)
    return a1 * relu(x - c1) + a2 * relu(x - c2) + (1.0 - a1 - a2) * relu(x - c3)


def derivative_levels(a):
    """Slope of h~ on its four segments (-inf,c1], (c1,c2], (c2,c3], (c3,inf).

    Each ReLU adds its weight to the slope once x passes its bias, so the slope
    on segment j is the sum of the first j weights. The weights sum to one, so the
    last slope is exactly 1.
    """
    a1, a2 = a
    return np.array([0.0, a1, a1 + a2, 1.0], dtype=np.float64)


def segment_code(x, c):
    """Segment index 0..3 of every element: how many biases lie strictly below x."""
    x = np.asarray(x, dtype=np.float64)
    if not np.all(np.isfinite(x)):
        raise ValueError("oracle inputs must be finite")
    c1, c2, c3 = c
    return ((x > c1).astype(np.uint8) + (x > c2).astype(np.uint8)
            + (x > c3).astype(np.uint8))


def gelu(x):
    """Exact GELU (Sec. 4.2): x/2 (1 + erf(x/sqrt2)), evaluated as x/2 erfc(-x/sqrt2).

    The two forms are equal since 1 + erf(u) = erfc(-u); the erfc form avoids the
    cancellation of 1 + erf for negative x.
    """
    x = np.asarray(x, dtype=np.float64)
    return 0.5 * x * erfc(-x / math.sqrt(2.0))


def silu(x):
    """Exact SiLU (Sec. 4.2): x / (1 + e^-x) = x * sigmoid(x)."""
    x = np.asarray(x, dtype=np.float64)
    return x * expit(x)


def codes_words(n):
    """Number of 32-bit words holding the 2-bit codes of n elements."""
    return (int(n) + 15) // 16


def pack_codes(codes):
    """Pack 2-bit codes of a flat sequence, 16 per uint32, least significant first."""
    codes = np.asarray(codes).reshape(-1)
    n = codes.size
    words = np.zeros(codes_words(n), dtype=np.uint32)
    for slot in range(16):
        part = codes[slot::16].astype(np.uint32)
        words[: part.size] |= part << np.uint32(2 * slot)
    return words


def unpack_codes(words, n):
    """Inverse of ``pack_codes``: the first n codes as uint8."""
    words = np.asarray(words, dtype=np.uint32).reshape(-1)
    if words.size != codes_words(n):
        raise ValueError("word count does not match n")
    out = np.empty(codes_words(n) * 16, dtype=np.uint8)
    for slot in range(16):
        out[slot::16] = (words >> np.uint32(2 * slot)) & np.uint32(3)
    return out[:n]


def _act_fwd(x, fn, c):
    x = np.asarray(x, dtype=np.float64)
    return fn(x), pack_codes(segment_code(x, c))


def _act_bwd(dy, words, a):
    dy = np.asarray(dy, dtype=np.float64)
    codes = unpack_codes(words, dy.size).reshape(dy.shape)
    return dy * derivative_levels(a)[codes]


def regelu2_fwd(x):
    """ReGELU2 forward: (GELU(x), packed segment codes for the GELU constants)."""
    return _act_fwd(x, gelu, GELU_C)


def regelu2_bwd(dy, words):
    """ReGELU2 backward: dy times the step derivative of h~ for the GELU constants."""
    return _act_bwd(dy, words, GELU_A)


def resilu2_fwd(x):
    """ReSiLU2 forward: (SiLU(x), packed segment codes for the SiLU constants)."""
    return _act_fwd(x, silu, SILU_C)


def resilu2_bwd(dy, words):
    """ReSiLU2 backward: dy times the step derivative of h~ for the SiLU constants."""
    return _act_bwd(dy, words, SILU_A)


# ---------------------------------------------------------------- SwiGLU

def reswiglu2_fwd(g, u):
    """ReSiLU2 inside a SwiGLU product (the LLaMA MLP, where the paper substitutes
    ReSiLU2 for SiLU, Sec. 6): s = SiLU(g), h = s * u, plus the 2-bit codes of g.

    Returns (h, s, packed codes). s is what the product's backward needs; SiLU's own
    backward needs only the codes (Sec. 4.2).
    """
    g = np.asarray(g, dtype=np.float64)
    u = np.asarray(u, dtype=np.float64)
    if g.shape != u.shape:
        raise ValueError("g and u must have the same shape")
    s = silu(g)
    return s * u, s, pack_codes(segment_code(g, SILU_C))


def reswiglu2_bwd(dh, u, s, words):
    """Approximate backward of h = SiLU(g) * u (Sec. 4.1: the backward of the network
    with h~ in place of SiLU, evaluated on the exact forward activations):
    du = dh * s (the exact product rule, s = SiLU(g) from the forward),
    dg = dh * u * slope of h~ at g (from the codes)."""
    dh = np.asarray(dh, dtype=np.float64)
    u = np.asarray(u, dtype=np.float64)
    s = np.asarray(s, dtype=np.float64)
    codes = unpack_codes(words, dh.size).reshape(dh.shape)
    return dh * u * derivative_levels(SILU_A)[codes], dh * s
