"""Pins for the oracle's DOT, FM, LayerNorm and MLP definitions."""
import numpy as np
import pytest

from oracle import interact, mlp
from oracle.bf16 import identity


def _naive_gram(Xb):
    n, d = Xb.shape
    Z = np.zeros((n, n))
    for i in range(n):
        for j in range(n):
            s = 0.0
            for a in range(d):
                s += Xb[i, a] * Xb[j, a]
            Z[i, j] = s
    return Z


def test_dot_matches_naive_upper_triangle_in_row_major_order():
    r = np.random.default_rng(0)
    B, n, d = 3, 5, 4
    X = r.standard_normal((B, n, d))
    p = interact.dot_forward(X, identity)
    assert p.shape == (B, n * (n - 1) // 2)
    for b in range(B):
        Z = _naive_gram(X[b])
        assert np.allclose(Z, Z.T)
        m = 0
        for i in range(n):
            for j in range(i + 1, n):
                # m(i,j) = i*n - i(i+1)/2 + (j-i-1)
                assert m == i * n - i * (i + 1) // 2 + (j - i - 1)
                assert abs(p[b, m] - Z[i, j]) < 1e-12
                m += 1


def test_dot_two_vectors_and_zero_slots():
    X = np.array([[[1.0, 2.0, 3.0], [4.0, -5.0, 6.0], [0.0, 0.0, 0.0]]])
    p = interact.dot_forward(X, identity)
    # pairs (0,1), (0,2), (1,2); slot 2 is an absent (zero-padded) feature
    np.testing.assert_array_equal(p, [[1 * 4 - 2 * 5 + 3 * 6, 0.0, 0.0]])


def test_dot_backward_matches_directional_derivative():
    # d/dt <p(X + tV), dp> at t=0 equals <dX, V>; p is quadratic so the
    # central difference is exact up to rounding
    r = np.random.default_rng(1)
    X, V = r.standard_normal((2, 6, 3)), r.standard_normal((2, 6, 3))
    dp = r.standard_normal((2, 15))
    dX = interact.dot_backward(dp, X)
    h = 1e-3
    fd = ((interact.dot_forward(X + h * V, identity) - interact.dot_forward(X - h * V, identity)) * dp).sum() / (2 * h)
    assert abs(fd - (dX * V).sum()) < 1e-9 * max(1.0, abs(fd))


def test_fm_identity_projection_is_full_gram():
    r = np.random.default_rng(2)
    B, n, d = 2, 5, 7
    X = r.standard_normal((B, n, d))
    O, _ = interact.fm_forward(X, np.eye(n), identity)
    for b in range(B):
        np.testing.assert_allclose(O[b], _naive_gram(X[b]), atol=1e-12)


def test_fm_unit_column_selects_gram_column():
    r = np.random.default_rng(3)
    X = r.standard_normal((1, 4, 3))
    W = np.zeros((4, 1))
    W[2, 0] = 1.0
    O, _ = interact.fm_forward(X, W, identity)
    np.testing.assert_allclose(O[0, :, 0], _naive_gram(X[0])[:, 2], atol=1e-12)


def test_fm_associativity():
    # X (X^T W) == (X X^T) W up to float64 rounding
    r = np.random.default_rng(4)
    X = r.standard_normal((3, 9, 16))
    W = r.standard_normal((9, 4))
    O, _ = interact.fm_forward(X, W, identity)
    for b in range(3):
        np.testing.assert_allclose(O[b], _naive_gram(X[b]) @ W, rtol=1e-12, atol=1e-12)


def test_layernorm_invariants():
    r = np.random.default_rng(5)
    u = r.standard_normal((4, 3, 16)) * 3 + 1.5
    y, xhat, _ = interact.layernorm_forward(u, np.ones(16), 0.0)
    np.testing.assert_allclose(y.mean(-1), 0, atol=1e-12)
    np.testing.assert_allclose((y ** 2).mean(-1), 1, atol=1e-12)
    # invariant to adding a constant to each vector
    y2, _, _ = interact.layernorm_forward(u + 7.25, np.ones(16), 0.0)
    np.testing.assert_allclose(y2, y, atol=1e-12)
    # gain scales the output per coordinate
    g = r.standard_normal(16)
    y3, _, _ = interact.layernorm_forward(u, g, 0.0)
    np.testing.assert_allclose(y3, y * g, atol=1e-12)


def test_linear_and_relu_against_triple_loop():
    r = np.random.default_rng(6)
    B, i, o = 4, 5, 3
    h = r.standard_normal((B, i))
    W, b = r.standard_normal((o, i)), r.standard_normal(o)
    hs, _ = mlp.mlp_forward(h, [(W, b)], identity, relu_last=True)
    for bb in range(B):
        for oo in range(o):
            s = b[oo]
            for ii in range(i):
                s += W[oo, ii] * h[bb, ii]
            assert abs(hs[1][bb, oo] - max(s, 0.0)) < 1e-12
    hs2, _ = mlp.mlp_forward(h, [(W, b)], identity, relu_last=False)
    assert np.any(hs2[1] < 0)                             # last layer is linear when asked


def test_linear_grads_against_loops():
    r = np.random.default_rng(7)
    B, i, o = 3, 4, 2
    h, g, W = r.standard_normal((B, i)), r.standard_normal((B, o)), r.standard_normal((o, i))
    dW, db, dh = mlp.linear_grads(g, h, W)
    for oo in range(o):
        for ii in range(i):
            assert abs(dW[oo, ii] - sum(g[bb, oo] * h[bb, ii] for bb in range(B))) < 1e-12
        assert abs(db[oo] - sum(g[bb, oo] for bb in range(B))) < 1e-12
    for bb in range(B):
        for ii in range(i):
            assert abs(dh[bb, ii] - sum(g[bb, oo] * W[oo, ii] for oo in range(o))) < 1e-12


def test_relu_override_only_moves_decisions_inside_the_band():
    r = np.random.default_rng(8)
    h = r.standard_normal((6, 5))
    W, b = r.standard_normal((4, 5)), r.standard_normal(4)
    a = mlp.linear(h, W, b)
    band = mlp.relu_band(h, W, b)
    assert np.all(band > 0) and np.all(band < 1e-5 * np.abs(h).sum(1).max() * 10)
    where = np.zeros_like(a, bool)
    where[0, 0] = True
    hs, m = mlp.mlp_forward(h, [(W, b)], identity, relu_last=True,
                            overrides=[(where, np.full_like(where, a[0, 0] <= 0))])
    ref, mref = mlp.mlp_forward(h, [(W, b)], identity, relu_last=True)
    assert m[0][0, 0] != mref[0][0, 0]
    assert hs[1][0, 0] == max(a[0, 0], 0.0) * m[0][0, 0]
    np.testing.assert_array_equal(np.delete(hs[1].ravel(), 0), np.delete(ref[1].ravel(), 0))
    np.testing.assert_array_equal(np.delete(m[0].ravel(), 0), np.delete(mref[0].ravel(), 0))
