"""Other members of the ReLU-combination family, in float64 (eq. relus_family for
general k; Appendix I). Test infrastructure only (see the package docstring).

* General k: 2^k - 1 ReLUs, weights a_1..a_{2^k-2} and last weight 1 - sum(a), biases
  c_1 < ... < c_{2^k-1}. The derivative is a 2^k-segment step function (Prop. 4.3), so
  a code of k bits per element selects the slope; slope on segment j is the sum of the
  first j weights.
* ReGELU2-d (Appendix I): k = 2 constants fitted to GELU's derivative instead of GELU.
* Packing: k bits per element, floor(32/k) codes per 32-bit word, least significant
  first (k in {1, 2, 3, 4}; for k = 3 that is 10 codes and the word's top two bits are
  zero, so no code straddles two words).
"""

import numpy as np

from .activations import codes_words as _words2, gelu, silu

# Appendix I: ReGELU2-d, the solution of the derivative-matching objective.
REGELU2D_A = (0.32465931184406527, 0.34812875668739607)
REGELU2D_C = (-0.4535743722857079, -0.0010587205574873046, 0.4487575313884231)


def relu_family(x, a, c):
    """h~_{a,c}(x) = sum_i a_i ReLU(x - c_i) + (1 - sum a) ReLU(x - c_last)."""
    x = np.asarray(x, dtype=np.float64)
    a = list(a)
    w = a + [1.0 - sum(a)]
    if len(w) != len(c):
        raise ValueError("need len(a) + 1 == len(c)")
    return sum(wi * np.maximum(x - ci, 0.0) for wi, ci in zip(w, c))


def family_levels(a):
    """Slopes of h~ on its len(a) + 2 segments: cumulative sums of the weights; the
    last one is exactly 1."""
    a = list(a)
    return np.array([0.0] + list(np.cumsum(a)) + [1.0], dtype=np.float64)


def family_code(x, c):
    """Number of biases strictly below x."""
    x = np.asarray(x, dtype=np.float64)
    if not np.all(np.isfinite(x)):
        raise ValueError("oracle inputs must be finite")
    return sum((x > ci).astype(np.uint8) for ci in c)


def words_for(bits, n):
    per = 32 // bits
    return (int(n) + per - 1) // per


def pack_bits(codes, bits):
    """k-bit codes, floor(32/k) per uint32 word, least significant first, zero tail."""
    if bits not in (1, 2, 3, 4):
        raise ValueError("bits must be 1, 2, 3 or 4")
    codes = np.asarray(codes).reshape(-1)
    per = 32 // bits
    words = np.zeros(words_for(bits, codes.size), dtype=np.uint32)
    for slot in range(per):
        part = codes[slot::per].astype(np.uint32)
        words[: part.size] |= part << np.uint32(bits * slot)
    return words


def unpack_bits(words, bits, n):
    per = 32 // bits
    words = np.asarray(words, dtype=np.uint32).reshape(-1)
    out = np.empty(words.size * per, dtype=np.uint8)
    for slot in range(per):
        out[slot::per] = (words >> np.uint32(bits * slot)) & np.uint32((1 << bits) - 1)
    return out[:n]


def stepact_fwd(x, act, c, bits):
    """Exact activation (``act`` in {"gelu", "silu"}) and packed k-bit codes."""
    if len(c) != (1 << bits) - 1:
        raise ValueError("need 2^bits - 1 biases")
    x = np.asarray(x, dtype=np.float64)
    y = gelu(x) if act == "gelu" else silu(x)
    return y, pack_bits(family_code(x, c), bits)


def stepact_bwd(dy, words, levels, bits):
    """dy times levels[code]."""
    dy = np.asarray(dy, dtype=np.float64)
    codes = unpack_bits(words, bits, dy.size).reshape(dy.shape)
    return dy * np.asarray(levels, dtype=np.float64)[codes]
