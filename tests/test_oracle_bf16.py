"""Pins for the oracle's float64 -> bfloat16 rounding."""
import numpy as np
import torch

from oracle.bf16 import round_bf16


def test_hand_cases_ties_to_even():
    one_ulp = 2.0 ** -7
    # exactly half an ulp above 1.0: tie -> even mantissa (1.0)
    assert round_bf16(1.0 + one_ulp / 2) == 1.0
    # 1 + 1.5 ulp: tie between 1+ulp (odd) and 1+2ulp (even) -> 1+2ulp
    assert round_bf16(1.0 + 1.5 * one_ulp) == 1.0 + 2 * one_ulp
    # a hair above the tie rounds up
    assert round_bf16(1.0 + one_ulp / 2 + 2.0 ** -30) == 1.0 + one_ulp
    # representable values are fixed points, sign symmetric
    for v in [0.0, -1.5, 3.0, 2.0 ** -126, 2.0 ** -133, 65280.0, -0.0078125]:
        assert round_bf16(v) == v
        assert round_bf16(-v) == -v
    # mantissa carry into the exponent: (2 - ulp/4) rounds to 2
    assert round_bf16(2.0 - one_ulp / 4) == 2.0
    # overflow beyond max + half ulp
    assert np.isinf(round_bf16(3.4e38))


def test_matches_torch_on_fp32_inputs():
    # torch's conversion is an independent implementation of the same rule
    r = np.random.default_rng(0)
    x = r.standard_normal(200_000) * np.exp(r.uniform(-80, 80, 200_000))
    x32 = x.astype(np.float32).astype(np.float64)
    ref = torch.from_numpy(x32.astype(np.float32)).to(torch.bfloat16).double().numpy()
    np.testing.assert_array_equal(round_bf16(x32), ref)


def test_result_is_nearest_grid_point():
    # brute force: the result is a bf16 value and no bf16 value is closer
    r = np.random.default_rng(1)
    x = r.uniform(0.5, 4.0, 5000)
    y = round_bf16(x)
    e = np.floor(np.log2(y))
    step = 2.0 ** (e - 7)
    assert np.all(np.abs(y / step - np.round(y / step)) == 0)
    assert np.all(np.abs(x - y) <= step / 2 + 1e-300)
