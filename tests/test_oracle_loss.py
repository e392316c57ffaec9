"""Pins for the oracle's masked multi-objective BCE."""
import math

import numpy as np

from oracle.loss import masked_bce, sigmoid


def test_zero_logits_give_log2():
    z = np.zeros((4, 3))
    y = np.array([[1, 0, 1], [0, 0, 1], [1, 1, 1], [0, 1, 0]], float)
    m = np.ones((4, 3))
    loss, dz = masked_bce(z, y, m)
    assert abs(loss - math.log(2.0)) < 1e-15
    np.testing.assert_allclose(dz, (0.5 - y) / 12, atol=1e-17)


def test_matches_textbook_cross_entropy():
    # -[y log s + (1-y) log(1-s)] with s = 1/(1+e^-z), evaluated naively at moderate z
    r = np.random.default_rng(0)
    z = r.uniform(-8, 8, (50, 4))
    y = (r.random((50, 4)) < 0.3).astype(float)
    m = (r.random((50, 4)) < 0.5).astype(float)
    s = 1.0 / (1.0 + np.exp(-z))
    naive = -(y * np.log(s) + (1 - y) * np.log(1 - s))
    loss, dz = masked_bce(z, y, m)
    assert abs(loss - (m * naive).sum() / m.sum()) < 1e-12
    np.testing.assert_allclose(dz, m * (s - y) / m.sum(), rtol=1e-12, atol=1e-18)


def test_large_logits_are_finite_and_asymptotic():
    z = np.array([[800.0, -800.0]])
    y = np.array([[0.0, 1.0]])
    loss, dz = masked_bce(z, y, np.ones((1, 2)))
    assert abs(loss - 800.0) < 1e-9                        # l(z,0) -> z, l(-z,1) -> z
    np.testing.assert_allclose(dz, [[0.5, -0.5]], atol=1e-15)


def test_all_masked_is_exactly_zero():
    r = np.random.default_rng(1)
    z = r.standard_normal((6, 5))
    loss, dz = masked_bce(z, np.ones((6, 5)), np.zeros((6, 5)))
    assert loss == 0.0
    assert np.all(dz == 0.0)


def test_masked_entries_have_exactly_zero_gradient():
    r = np.random.default_rng(2)
    z = r.standard_normal((10, 4))
    y = (r.random((10, 4)) < 0.5).astype(float)
    m = (r.random((10, 4)) < 0.5).astype(float)
    _, dz = masked_bce(z, y, m)
    assert np.all(dz[m == 0] == 0.0)
    # and the loss does not depend on masked logits at all
    z2 = z.copy()
    z2[m == 0] += 100.0
    assert masked_bce(z2, y, m)[0] == masked_bce(z, y, m)[0]


def test_label_symmetry_and_sigmoid():
    z = np.linspace(-5, 5, 11)[None]
    l1, _ = masked_bce(z, np.ones_like(z), np.ones_like(z))
    l0, _ = masked_bce(-z, np.zeros_like(z), np.ones_like(z))
    assert abs(l1 - l0) < 1e-14
    np.testing.assert_allclose(sigmoid(z) + sigmoid(-z), 1.0, atol=1e-15)
