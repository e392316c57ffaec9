"""Masked multi-objective binary cross-entropy.

Test infrastructure only (see the package docstring).

Every sample produces one logit per objective (Section 3.3); an impression
trains only the heads it is routed to (Section 3.2.1), which is a 0/1 mask
``m[b, t]``.  With ``N = max(1, sum m)``:

    l(z, y) = max(z, 0) - z*y + log1p(exp(-|z|))     (BCE with logits, stable form)
    L       = sum_{b,t} m*l / N
    dL/dz   = m * (sigmoid(z) - y) / N

so masked entries contribute exactly zero loss and gradient.
"""
import numpy as np


def sigmoid(z):
    z = np.asarray(z, np.float64)
    e = np.exp(-np.abs(z))
    return np.where(z >= 0, 1.0 / (1.0 + e), e / (1.0 + e))


def masked_bce(z, y, m, normalizer=None):
    """(loss, dz) in float64.  ``normalizer`` replaces ``max(1, sum m)`` when
    the rows given are a subset of a larger batch whose labelled-entry count
    defines N."""
    z = np.asarray(z, np.float64)
    y = np.asarray(y, np.float64)
    m = np.asarray(m, np.float64)
    N = max(1.0, float(m.sum())) if normalizer is None else float(normalizer)
    l = np.maximum(z, 0.0) - z * y + np.log1p(np.exp(-np.abs(z)))
    loss = float((m * l).sum() / N)
    dz = m * (sigmoid(z) - y) / N
    return loss, dz
