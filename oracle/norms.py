"""MS-LN and MS-RMSNorm in float64 (Sec. 5.2 Alg. 1; Appendix G Alg. 2 and Alg. 3).

Test infrastructure only (see the package docstring).

With the affine (alpha, beta) merged into the following linear layer
(W~ = W diag(alpha), b~ = W beta + b, Sec. 5.2), a normalisation layer has no
parameters, and its Jacobian can be written with its own output z and the scalar
sigma. Forward and backward for a row x of width p:

    sigma = sqrt(p^-1 x^T H^T H x + eps),   z = sigma^-1 H x,
    dx    = sigma^-1 (H - p^-1 z z^T) dz,

with H = I - p^-1 1 1^T for LayerNorm and H = I for RMSNorm. Applying H to a
vector subtracts its mean; the oracle writes that product out elementwise rather
than forming the p x p matrix.

Readings where the paper leaves a choice open:

* The saved statistic is rstd = 1/sigma (the paper saves sigma; only its inverse is
  ever used). It is produced here in float64; stored copies are fp32.
* The backward uses the Appendix G form sigma^-1 (H - p^-1 z z^T) dz. The Sec. 5.2
  form sigma^-1 H^T (I - p^-1 z z^T) dz is equal whenever H z = z, i.e. whenever z
  has zero mean, which holds for the exact forward output.
* The backward consumes the z and rstd it is given (the stored values), not a
  recomputation from x.
"""

import numpy as np


def _rows(a):
    a = np.asarray(a, dtype=np.float64)
    if a.ndim != 2:
        raise ValueError("norm inputs are 2-D [rows, p]")
    if not np.all(np.isfinite(a)):
        raise ValueError("oracle inputs must be finite")
    return a


def _center(v):
    """H v for LayerNorm: v minus its row mean."""
    return v - v.mean(axis=1, keepdims=True)


def _fwd(x, eps, centered):
    x = _rows(x)
    p = x.shape[1]
    hx = _center(x) if centered else x
    sigma = np.sqrt((hx * hx).sum(axis=1) / p + float(eps))
    rstd = 1.0 / sigma
    z = hx * rstd[:, None]
    return z, rstd


def _bwd(dz, z, rstd, centered):
    dz = _rows(dz)
    z = _rows(z)
    rstd = np.asarray(rstd, dtype=np.float64).reshape(-1)
    if dz.shape != z.shape or rstd.size != z.shape[0]:
        raise ValueError("shape mismatch")
    p = z.shape[1]
    h_dz = _center(dz) if centered else dz
    proj = z * ((z * dz).sum(axis=1, keepdims=True) / p)   # p^-1 z (z^T dz)
    return rstd[:, None] * (h_dz - proj)


def msln_fwd(x, eps):
    """MS-LN forward (Alg. 1 / Alg. 2): returns (z, rstd) for rows of x."""
    return _fwd(x, eps, centered=True)


def msln_bwd(dz, z, rstd):
    """MS-LN backward (Alg. 2): dx = rstd * (H - p^-1 z z^T) dz."""
    return _bwd(dz, z, rstd, centered=True)


def msrms_fwd(x, eps):
    """MS-RMSNorm forward (Alg. 3): returns (z, rstd) with H = I."""
    return _fwd(x, eps, centered=False)


def msrms_bwd(dz, z, rstd):
    """MS-RMSNorm backward (Alg. 3): dx = rstd * (I - p^-1 z z^T) dz."""
    return _bwd(dz, z, rstd, centered=False)
