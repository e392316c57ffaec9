"""Pins for the e4m3 quantiser and FP8 linear layer of ``oracle.fp8``:
torch's float8_e4m3fn conversion (an independent implementation of the same
OCP format) bit for bit, the round trip of every finite code, ties to even
at every midpoint, saturation, the per-row / per-tensor scale rule, and the
dequantised product against a triple loop."""
import numpy as np
import pytest
import torch

from oracle import fp8


def test_codes_match_torch_float8_e4m3fn():
    rng = np.random.default_rng(0)
    v = np.concatenate([
        rng.standard_normal(20000) * np.exp2(rng.integers(-14, 9, 20000)),
        rng.uniform(-464, 464, 5000),                      # up to the saturation tie
        [0.0, -0.0, 448.0, -448.0, 2.0 ** -6, 2.0 ** -9, 2.0 ** -10, 3 * 2.0 ** -11, 1e-30],
    ]).astype(np.float32)
    v = v[np.abs(v) <= 464]
    ref = torch.from_numpy(v).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    np.testing.assert_array_equal(fp8.e4m3_code(v), ref)


def test_every_finite_code_round_trips_and_midpoints_tie_to_even():
    codes = np.array([c for c in range(256) if (c & 0x7F) != 0x7F], np.uint8)
    vals = fp8.e4m3_value(codes)
    np.testing.assert_array_equal(fp8.e4m3_code(vals), codes)
    # torch agrees on the decoded values
    tv = torch.from_numpy(codes.copy()).view(torch.float8_e4m3fn).float().numpy()
    np.testing.assert_array_equal(tv, vals.astype(np.float32))
    pos = np.sort(np.unique(vals[vals >= 0]))
    mids = (pos[:-1] + pos[1:]) / 2
    got = fp8.e4m3_value(fp8.e4m3_code(mids))
    lo, hi = pos[:-1], pos[1:]
    lo_even = (fp8.e4m3_code(lo).astype(int) & 1) == 0
    np.testing.assert_array_equal(got, np.where(lo_even, lo, hi))


def test_saturation_and_signs():
    assert fp8.e4m3_code(np.array([470.0, 1e6, -1e6])).tolist() == [0x7E, 0x7E, 0xFE]
    assert fp8.e4m3_code(np.array([-0.0, 0.0, -1e-30])).tolist() == [0x80, 0x00, 0x80]


@pytest.mark.parametrize("rowwise", [True, False])
def test_quantize_scale_rule(rowwise):
    rng = np.random.default_rng(1)
    x = (rng.standard_normal((40, 77)) * np.exp2(rng.integers(-8, 8, (40, 1)))).astype(np.float32)
    x[3] = 0.0                                            # an all-zero row: scale 1, codes 0
    q, s = fp8.quantize(x, rowwise)
    assert q.shape == x.shape and s.dtype == np.float32
    amax = np.abs(x).max(1) if rowwise else np.array([np.abs(x).max()])
    np.testing.assert_array_equal(s, np.where(amax > 0, (amax / np.float32(448)).astype(np.float32), 1))
    vals = fp8.e4m3_value(q)
    # the largest magnitude of each row / of the tensor maps to +-448
    if rowwise:
        nz = amax > 0
        np.testing.assert_array_equal(np.abs(vals).max(1)[nz], 448.0)
        assert not np.any(q[3])
    else:
        assert np.abs(vals).max() == 448.0
    # a power-of-two scaling of the input scales the scales, not the codes
    q2, s2 = fp8.quantize(x * np.float32(8.0), rowwise)
    np.testing.assert_array_equal(q2, q)
    np.testing.assert_array_equal(s2[s2 != 1], (s * 8)[s2 != 1])
    # dequantised values within half an e4m3 step (relative 2^-4) of x
    deq = fp8.dequantize(q, s, rowwise)
    big = np.abs(x / (s[:, None] if rowwise else s[0])) >= 2 ** -6
    assert np.all(np.abs(deq - x)[big] <= 2.0 ** -4 * np.abs(x)[big] * (1 + 1e-6))


def test_linear_fp8_against_triple_loop():
    rng = np.random.default_rng(2)
    x = rng.standard_normal((5, 9)).astype(np.float32)
    w = rng.standard_normal((4, 9)).astype(np.float32)
    b = rng.standard_normal(4)
    qa, sa = fp8.quantize(x, True)
    qw, sw = fp8.quantize(w, True)
    y = fp8.linear_fp8(qa, sa, qw, sw, b, relu=True)
    A, W = fp8.e4m3_value(qa), fp8.e4m3_value(qw)
    for m in range(5):
        for n in range(4):
            s = sum(A[m, k] * W[n, k] for k in range(9))
            assert abs(y[m, n] - max(s * sa[m] * sw[n] + b[n], 0.0)) < 1e-12
    qt, st = fp8.quantize(x, False)
    yt = fp8.linear_fp8(qt, st, qw, sw)
    np.testing.assert_allclose(yt, (fp8.e4m3_value(qt) * st[0]) @ (W * sw[:, None]).T, rtol=1e-13)


@pytest.mark.parametrize("fast", [False, True])
def test_product_bound_covers_aligned_accumulation(fast):
    """The accepted deviation of an FP8 product covers an evaluation whose
    matrix instruction truncates every addend to 13 fraction bits of the
    step's largest exponent (the behaviour measured on the accelerator),
    with the partial sum chained through K (fast) or restarted per step."""
    rng = np.random.default_rng(3)
    x = (rng.standard_normal((6, 300)) * np.exp2(rng.integers(-6, 3, (6, 300)))).astype(np.float32)
    w = rng.standard_normal((5, 300)).astype(np.float32)
    qa, sa = fp8.quantize(x, True)
    qw, sw = fp8.quantize(w, True)
    A, W = fp8.e4m3_value(qa), fp8.e4m3_value(qw)
    exact = A @ W.T
    emu = np.zeros_like(exact)
    for m in range(6):
        for n in range(5):
            acc = 0.0
            for k0 in range(0, 300, 64):
                p = A[m, k0:k0 + 64] * W[n, k0:k0 + 64]
                if fast:
                    acc = fp8.emulate_aligned_sum(p, acc)
                else:
                    acc = float(np.float32(acc + np.float32(fp8.emulate_aligned_sum(p))))
            emu[m, n] = acc
    bound = fp8.linear_fp8_bound(qa, np.ones(6), qw, np.ones(5), fast_accum=fast)
    assert np.any(emu != exact)
    assert np.all(np.abs(emu - exact) <= bound)
    # restarting every step keeps the bound a small fraction of the sum of
    # magnitudes; chaining the partial sum makes it grow with K
    frac = bound / (np.abs(A) @ np.abs(W).T)
    assert np.all(frac <= (0.05 if fast else 0.01))
