"""Pins of the per-objective towers' heads (Section 3.3.3): objective t's
logit reads only its tower's hidden units, so the grouped layer is the dense
linear layer whose weight is block-diagonal -- row t zero outside columns
t*H .. t*H+H-1 -- and its gradients are the dense gradients restricted to
those blocks."""
import numpy as np

from oracle import mlp


def _block_diag(W):
    T, H = W.shape
    Wf = np.zeros((T, T * H))
    for t in range(T):
        Wf[t, t * H:(t + 1) * H] = W[t]
    return Wf


def test_grouped_heads_are_a_block_diagonal_dense_layer():
    rng = np.random.default_rng(5)
    B, T, H = 7, 4, 3
    h = rng.standard_normal((B, T * H))
    W = rng.standard_normal((T, H))
    b = rng.standard_normal(T)
    a = mlp.grouped_linear(h, W, b)
    assert np.max(np.abs(a - mlp.linear(h, _block_diag(W), b))) < 1e-13
    # brute force for one element
    t, r = 2, 5
    assert abs(a[r, t] - (sum(h[r, t * H + j] * W[t, j] for j in range(H)) + b[t])) < 1e-13
    g = rng.standard_normal((B, T))
    dW, db, dh = mlp.grouped_linear_grads(g, h, W)
    dWf, dbf, dhf = mlp.linear_grads(g, h, _block_diag(W))
    assert np.max(np.abs(dh - dhf)) < 1e-13 and np.max(np.abs(db - dbf)) < 1e-13
    for t in range(T):
        assert np.max(np.abs(dW[t] - dWf[t, t * H:(t + 1) * H])) < 1e-13
