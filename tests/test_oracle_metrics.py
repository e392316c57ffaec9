"""Pins for the comparison metrics that decide every parity test
(``oracle.metrics``) and for the ReLU ambiguity band (``oracle.mlp.relu_band``).

The metrics are checked on hand-computed inputs; the band against fp32
summation carried out in many orders (numpy float32 arithmetic, one addition
at a time), which is what the band claims to bound."""
import itertools

import numpy as np
import pytest

from oracle import mlp
from oracle.metrics import max_rel_err, max_rel_err_normwise


# ---------------------------------------------------------------- max_rel_err
def test_rel_err_hand_computed_rows():
    r = np.array([[3.0, 4.0], [1.0, -1.0]])
    # row 0: rms = sqrt((9+16)/2) = 3.5355...; element 0 is normalised by
    # max(3, 3.5355) = 3.5355, element 1 by 4
    x = np.array([[3.5, 4.0], [1.0, -1.0]])
    assert max_rel_err(x, r) == pytest.approx(0.5 / np.sqrt(12.5), rel=1e-15)
    x = np.array([[3.0, 4.4], [1.0, -1.0]])
    assert max_rel_err(x, r) == pytest.approx(0.4 / 4.0, rel=1e-14)
    # row 1: rms 1, |r| 1
    x = np.array([[3.0, 4.0], [1.0, -1.25]])
    assert max_rel_err(x, r) == pytest.approx(0.25, rel=1e-15)


def test_rel_err_tiny_element_is_normalised_by_its_row_rms():
    # a reference element that is small only by cancellation must not be
    # judged by its own magnitude, but by the rms of its row
    r = np.array([[1e-6, 1.0, -1.0, 1.0]])
    x = r.copy()
    x[0, 0] += 1e-3                  # 1000x its own magnitude, 1e-3 of the row rms
    assert max_rel_err(x, r) == pytest.approx(1e-3 / np.sqrt((1e-12 + 3) / 4), rel=1e-9)
    assert max_rel_err(x, r) < 2e-2
    # the same absolute error in a row whose rms is 1e-6 fails
    r2 = np.array([[1e-6, 1e-6]])
    assert max_rel_err(r2 + np.array([[1e-3, 0.0]]), r2) > 100


def test_rel_err_zero_reference_row_demands_exact_zeros():
    r = np.array([[0.0, 0.0, 0.0], [1.0, 2.0, 3.0]])
    assert max_rel_err(r.copy(), r) == 0.0
    x = r.copy()
    x[0, 1] = 1e-30
    assert max_rel_err(x, r) == float("inf")
    x = r.copy()
    x[0, 2] = -0.0                   # negative zero is zero
    assert max_rel_err(x, r) == 0.0


def test_rel_err_non_finite_fails():
    r = np.ones((2, 3))
    for bad in (np.nan, np.inf, -np.inf):
        x = r.copy()
        x[1, 2] = bad
        assert max_rel_err(x, r) == float("inf")
        assert max_rel_err_normwise(x, r) == float("inf")


def test_rel_err_planted_error_fails_the_bf16_bound():
    rng = np.random.default_rng(3)
    r = rng.standard_normal((64, 128))
    x = r * (1 + 1e-3 * rng.standard_normal(r.shape))
    assert max_rel_err(x, r) < 2e-2
    # one element 3% off (relative to its row rms) in an otherwise exact tensor
    i, j = 17, 99
    rms = np.sqrt(np.mean(r[i] ** 2))
    x[i, j] = r[i, j] + 3e-2 * max(abs(r[i, j]), rms)
    assert max_rel_err(x, r) == pytest.approx(3e-2, rel=1e-9)
    assert max_rel_err(x, r) > 2e-2


def test_rel_err_scalars_and_vectors_use_the_whole_tensor():
    # 1-D: one "row"; rms over all elements
    r = np.array([0.0, 2.0])
    assert max_rel_err(np.array([0.1, 2.0]), r) == pytest.approx(0.1 / np.sqrt(2.0), rel=1e-15)
    assert max_rel_err(np.array(1.01), np.array(1.0)) == pytest.approx(0.01, rel=1e-12)
    assert max_rel_err(np.zeros((0, 4)), np.zeros((0, 4))) == 0.0
    with pytest.raises(ValueError):
        max_rel_err(np.zeros(3), np.zeros(4))


def test_rel_err_rows_are_the_last_axis():
    # a 3-D tensor: rows are the last-axis vectors, not the whole tensor
    r = np.ones((2, 3, 4))
    r[1, 2] = 1e-3                   # a small row
    x = r.copy()
    x[1, 2, 0] += 1e-3               # 100% of that row's rms
    assert max_rel_err(x, r) == pytest.approx(1.0, rel=1e-12)
    # judged against the whole tensor it would look like 1e-3
    assert max_rel_err(x.reshape(-1), r.reshape(-1)) < 2e-3


# ------------------------------------------------------- max_rel_err_normwise
def test_normwise_hand_computed():
    r = np.array([[1.0, -4.0], [0.5, 2.0]])
    x = np.array([[1.2, -4.0], [0.5, 2.0]])
    assert max_rel_err_normwise(x, r) == pytest.approx(0.2 / 4.0, rel=1e-14)
    # an error in the largest element counts the same as one in a small element
    x = np.array([[1.0, -4.2], [0.5, 2.0]])
    assert max_rel_err_normwise(x, r) == pytest.approx(0.2 / 4.0, rel=1e-14)
    assert max_rel_err_normwise(np.zeros(3), np.zeros(3)) == 0.0
    assert max_rel_err_normwise(np.array([0.0, 1e-300]), np.zeros(2)) == float("inf")
    # planted: 3% of the largest magnitude fails 2e-2
    x = r.copy()
    x[1, 0] += 0.03 * 4.0
    assert max_rel_err_normwise(x, r) > 2e-2


def test_normwise_is_never_stricter_than_elementwise():
    rng = np.random.default_rng(5)
    for _ in range(20):
        r = rng.standard_normal((8, 16)) * rng.uniform(0.01, 10, (8, 1))
        x = r + 1e-2 * rng.standard_normal(r.shape)
        assert max_rel_err_normwise(x, r) <= max_rel_err(x, r) * (1 + 1e-12)


# ----------------------------------------------------------------- relu_band
def _fp32_sums_in_orders(h, W, b, rng, n_orders):
    """fp32 evaluations of h.W + b, one addition at a time, in several orders
    (products rounded to fp32 first, as an fp32 FMA-free accumulation does,
    and fused, as an FMA chain does)."""
    K = h.size
    terms64 = h * W
    out = []
    orders = [np.arange(K), np.arange(K)[::-1]] + [rng.permutation(K) for _ in range(n_orders)]
    for order in orders:
        for fused in (False, True):
            s = np.float32(b)
            for k in order:
                if fused:      # fp32 FMA: exact product, one rounding of the sum
                    s = np.float32(np.float64(s) + terms64[k])
                else:
                    s = np.float32(s + np.float32(terms64[k]))
            out.append(float(s))
        # pairwise (tree) summation
        v = [np.float32(terms64[k]) for k in order] + [np.float32(b)]
        while len(v) > 1:
            v = [np.float32(v[i] + v[i + 1]) if i + 1 < len(v) else v[i] for i in range(0, len(v), 2)]
        out.append(float(v[0]))
    return np.array(out)


def test_relu_band_bounds_fp32_summation_in_any_order():
    rng = np.random.default_rng(11)
    worst = 0.0
    for trial in range(60):
        K = int(rng.integers(2, 24))
        # operands exactly representable in bf16 (as the GEMM operands are),
        # spread over several binades so that summation order matters
        h = np.float32(rng.standard_normal(K) * 2.0 ** rng.integers(-6, 6, K)).astype(np.float64)
        W = np.float32(rng.standard_normal(K) * 2.0 ** rng.integers(-6, 6, K)).astype(np.float64)
        if trial % 3 == 0:            # engineered cancellation: a tiny exact value
            h[-1] = -np.sum(h[:-1] * W[:-1]) / W[-1]
            h[-1] = float(np.float32(h[-1]))
        b = float(np.float32(rng.standard_normal() * 0.01))
        exact = float(np.sum(h * W) + b)
        band = float(mlp.relu_band(h[None], W[None], np.array([b]))[0, 0])
        sums = _fp32_sums_in_orders(h, W, b, rng, 6)
        err = np.abs(sums - exact).max()
        assert err <= band, (trial, err, band)
        worst = max(worst, err / band)
    # the band is not vacuous: the observed errors use a visible part of it
    assert worst > 1e-3


def test_relu_band_planted_mistakes_fail():
    # a crafted cancellation case whose fp32 sums land far from the exact value
    h = np.array([1.0, 2.0 ** -24, 2.0 ** -24, 2.0 ** -24, -1.0])
    W = np.array([1.0, 1.0, 1.0, 1.0, 1.0])
    b = 0.0
    exact = 3 * 2.0 ** -24
    rng = np.random.default_rng(0)
    err = np.abs(_fp32_sums_in_orders(h, W, b, rng, 10) - exact).max()
    assert err > 0
    band = mlp.relu_band(h[None], W[None], np.array([b]))[0, 0]
    assert err <= band
    # mistakes: absolute values dropped (the sum of signed terms), or the bound
    # taken per term (2^-24 * sum|terms| without the K factor)
    signed = (h.size + 1) * 2.0 ** -24 * abs(np.sum(h * W) + b)
    assert err > signed
    per_term = 2.0 ** -24 * (np.sum(np.abs(h * W)) + abs(b))
    h2 = np.array([1.0] + [2.0 ** -25] * 6 + [-1.0])
    W2 = np.ones_like(h2)
    err2 = np.abs(_fp32_sums_in_orders(h2, W2, 0.0, rng, 10) - 6 * 2.0 ** -25).max()
    per_term2 = 2.0 ** -24 * np.sum(np.abs(h2))
    assert err2 > per_term2
    assert err2 <= mlp.relu_band(h2[None], W2[None], np.zeros(1))[0, 0]
    assert per_term < band


@pytest.mark.parametrize("K", [1, 3, 8])
def test_relu_band_shapes_and_bias(K):
    rng = np.random.default_rng(K)
    h = rng.standard_normal((4, K))
    W = rng.standard_normal((5, K))
    b = rng.standard_normal(5)
    band = mlp.relu_band(h, W, b)
    assert band.shape == (4, 5)
    brute = np.zeros((4, 5))
    for i, j in itertools.product(range(4), range(5)):
        brute[i, j] = (K + 1) * 2.0 ** -24 * (sum(abs(h[i, k] * W[j, k]) for k in range(K)) + abs(b[j]))
    np.testing.assert_allclose(band, brute, rtol=1e-12)
