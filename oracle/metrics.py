"""Comparison metrics of the parity tests.

Test infrastructure only (see the package docstring).

``max_rel_err(x, r)`` is the largest ``|x_i - r_i| / max(|r_i|, rms(row_i(r)))``
over all elements, where ``row_i`` is the last-axis vector holding element i
(the whole tensor for scalars and 1-D tensors).  A row that is identically zero
in the reference must be exactly zero in ``x``; a non-finite value in ``x``
fails.  Normalising by the row's rms keeps elements that are tiny only by
cancellation from dominating a relative metric.
"""
import numpy as np


def max_rel_err(x, r):
    x = np.asarray(x, np.float64)
    r = np.asarray(r, np.float64)
    if x.shape != r.shape:
        raise ValueError(f"shape mismatch {x.shape} vs {r.shape}")
    if r.size == 0:
        return 0.0
    if not np.all(np.isfinite(x)):
        return float("inf")
    rr = r.reshape(1, -1) if r.ndim <= 1 else r.reshape(-1, r.shape[-1])
    xx = x.reshape(rr.shape)
    rms = np.sqrt(np.mean(rr * rr, axis=-1, keepdims=True))
    zero = rms[:, 0] == 0
    if np.any(xx[zero] != 0):
        return float("inf")
    denom = np.maximum(np.abs(rr), rms)
    ok = denom > 0
    err = np.zeros_like(rr)
    err[ok] = np.abs(xx[ok] - rr[ok]) / denom[ok]
    return float(err.max())


def max_rel_err_normwise(x, r):
    """Largest absolute deviation relative to the largest reference magnitude,
    ``max_i |x_i - r_i| / max_i |r_i|`` (0 for an all-zero reference that x
    matches exactly; a non-finite value in x fails)."""
    x = np.asarray(x, np.float64)
    r = np.asarray(r, np.float64)
    if x.shape != r.shape:
        raise ValueError(f"shape mismatch {x.shape} vs {r.shape}")
    if r.size == 0:
        return 0.0
    if not np.all(np.isfinite(x)):
        return float("inf")
    scale = np.abs(r).max()
    diff = np.abs(x - r).max()
    if scale == 0:
        return 0.0 if diff == 0 else float("inf")
    return float(diff / scale)
