"""Storage formats seen by the oracle: fp32 and bf16 (as raw uint16 bit patterns).

Test infrastructure only (see the package docstring).

The paper does not fix a storage precision for the kernels; its experiments run
the activations in 16-bit mixed precision and keep normalisation statistics in
fp32 (captions of the activation-memory figures, Appendix B). The oracle therefore
accepts the exact bytes a kernel consumes, decodes them to float64 without loss,
and can round float64 results back to either format with a single correct
round-to-nearest-even step.
"""

import numpy as np

DTYPES = ("fp32", "bf16")


def decode(arr, dtype):
    """Exact float64 value of stored elements.

    fp32: ``arr`` is a float32 array. bf16: ``arr`` holds the 16-bit patterns as
    uint16; a bf16 value is the fp32 value whose upper half is the pattern and whose
    lower half is zero, so widening is exact.
    """
    if dtype == "fp32":
        a = np.asarray(arr)
        if a.dtype != np.float32:
            raise TypeError("fp32 storage must be a float32 array")
        return a.astype(np.float64)
    if dtype == "bf16":
        a = np.asarray(arr)
        if a.dtype != np.uint16:
            raise TypeError("bf16 storage must be a uint16 array of bit patterns")
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    raise ValueError(f"unknown dtype {dtype!r}")


def _round_bf16_value(x):
    """Nearest bf16 value to each float64 in ``x`` (ties to even), as float64.

    bf16 keeps 8 significant bits and the fp32 exponent range. For |x| in
    [2^e, 2^(e+1)) the spacing of bf16 values is 2^(e-7); below the smallest
    normal 2^-126 the spacing stays 2^-133. Dividing by a power of two is exact, so
    ``rint`` (round half to even) on the scaled value is the rounding itself.
    """
    x = np.asarray(x, dtype=np.float64)
    _, e2 = np.frexp(x)               # x = m * 2^e2 with 0.5 <= |m| < 1
    e = np.maximum(e2 - 1, -126)      # floor(log2|x|), clamped at the subnormal range
    ulp = np.ldexp(1.0, e - 7)
    return np.rint(x / ulp) * ulp


def round_to_dtype(x, dtype):
    """float64 -> nearest value of ``dtype`` (RNE), returned as float64."""
    x = np.asarray(x, dtype=np.float64)
    if not np.all(np.isfinite(x)):
        raise ValueError("oracle values must be finite")
    if dtype == "fp32":
        return x.astype(np.float32).astype(np.float64)
    if dtype == "bf16":
        return _round_bf16_value(x)
    raise ValueError(f"unknown dtype {dtype!r}")


def encode(x, dtype):
    """float64 -> storage array of ``dtype`` holding the RNE-rounded values."""
    r = round_to_dtype(x, dtype)
    if dtype == "fp32":
        return r.astype(np.float32)
    # r is exactly representable in bf16, hence in fp32: take the upper 16 bits.
    return (r.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
