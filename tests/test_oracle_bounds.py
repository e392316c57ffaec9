"""Pins for the element-wise error scales of ``oracle.bounds``, the rule
that decides which differences between the accelerator's composed bf16 step
and the oracle are correct arithmetic.

The scales claim to cover any evaluation of the step that differs from the
oracle's only in accumulation order (fp32) and in which way values near a
rounding boundary round.  They are checked against such evaluations made on
the CPU: the oracle run again with every stored value perturbed before its
rounding by a random relative amount at the fp32 accumulation level, which
moves values across bf16 rounding boundaries exactly as a different fp32
summation order does.  A planted mistake in the propagation rules must make
that check fail, and the primitive rules are checked against brute force."""
import numpy as np
import pytest

import synth
from oracle import bf16, bounds, step

UA = 2.0 ** -24


def _perturbed_rounding(rng, amp):
    def r(x):
        x = np.asarray(x, np.float64)
        return bf16.round_bf16(x * (1 + amp * UA * rng.uniform(-1, 1, x.shape)))
    return r


CASES = {
    "mid-dot": lambda: synth.small(synth.MID, B=96, rows=400),
    "large-fm-sgd": lambda: synth.small(synth.LARGE_FM, B=32, rows=300),
    "multidomain-dot": lambda: synth.small(synth.MULTIDOMAIN, B=64, rows=300),
    "deep-stack": lambda: synth.DEEP_STACK.scaled(B=12, F=16, rows=300, d=32, stack_n=8, fm_rank=8,
                                                  top=(64, 16, 4)),
}


def _pairs(c, g, bd, c2, g2):
    """(name, perturbed, reference, scales) of every compared tensor."""
    out = [("X", c2["X"], c["X"], bd["X"]), ("t", c2["t"], c["t"], bd["t"]),
           ("logits", c2["logits"], c["logits"], bd["logits"]),
           ("loss", [c2["loss"]], [c["loss"]], bd["loss"]), ("dz", c2["dz"], c["dz"], bd["dz"]),
           ("d_top_in", g2["d_top_in"], g["d_top_in"], bd["d_top_in"]),
           ("dX_emb", g2["dX_emb"], g["dX_emb"], bd["dX_emb"]),
           ("grad_rows", g2["grad_rows"], g["grad_rows"], bd["grad_rows"])]
    for key in ("top_dW", "top_db", "bottom_dW", "bottom_db"):
        for i, e in enumerate(bd.get(key, [])):
            out.append((f"{key}{i}", g2[key][i], g[key][i], e))
    if "fm_dW" in bd:
        out.append(("fm_dW", g2["fm_dW"], g["fm_dW"], bd["fm_dW"]))
    for l, gl in enumerate(bd.get("stack", [])):
        for k, e in gl.items():
            out.append((f"stack{l}.{k}", g2["stack"][l][k], g["stack"][l][k], e))
    if "updated_rows" in bd:
        out.append(("updated_rows", g2["updated_rows"], g["updated_rows"], bd["updated_rows"]))
    return out


def _worst_ratio(name, seeds=(0, 1)):
    cfg = CASES[name]()
    batch = synth.make_batch(cfg)
    params = synth.make_dense_params(cfg)
    table = synth.make_tables(cfg).double().numpy()
    c, g = step.step(cfg, params, table, batch)
    bd = bounds.step_bounds(cfg, params, table, batch, c, g)
    worst, moved = {}, 0
    orig = step.rounding
    for seed in seeds:
        rng = np.random.default_rng(seed)
        step.rounding = lambda dt: _perturbed_rounding(rng, 4.0) if dt == "bf16" else bf16.identity
        try:
            c2, g2 = step.step(cfg, params, table, batch)
        finally:
            step.rounding = orig
        for k, a, b, e in _pairs(c, g, bd, c2, g2):
            diff = np.abs(np.asarray(a, np.float64) - np.asarray(b, np.float64))
            moved += int(np.count_nonzero(diff))
            worst[k] = max(worst.get(k, 0.0), float((diff / (bounds.allowed(e) + 1e-300)).max()))
    return worst, moved, bd, c


@pytest.mark.parametrize("name", list(CASES))
def test_scales_cover_evaluations_that_round_differently(name):
    worst, moved, _, _ = _worst_ratio(name)
    assert moved > 1000                     # the perturbation does flip many roundings
    bad = {k: v for k, v in worst.items() if v > 1.0}
    assert not bad, bad


def test_scales_are_not_vacuous_where_nothing_cancels():
    # values rounded once from well-conditioned sums (the pooled lookups):
    # the accepted deviation is a few bf16 ulps, i.e. a few percent at most
    _, _, bd, c = _worst_ratio("mid-dot", seeds=())
    s0 = 1
    acc = bounds.allowed(bd["X"])[:, s0:]
    ref = np.abs(c["X"][:, s0:])
    nz = ref > 0
    ratio = acc[nz] / ref[nz]
    assert np.median(ratio) < 0.03 and np.quantile(ratio, 0.9) < 0.05


def test_planted_mistake_in_the_rounding_rule_fails_the_cover(monkeypatch):
    """Without the jump a rounding can add, evaluations that round the other
    way fall outside the scales."""
    def no_jump(e, y, us):
        s, m = e
        return np.sqrt(s * s + 6.0 * us * np.abs(y) * s), m * (1.0 + us)
    monkeypatch.setattr(bounds, "rounded", no_jump)
    worst, _, _, _ = _worst_ratio("mid-dot", seeds=(0,))
    assert max(worst.values()) > 1.0


def test_planted_mistake_in_the_product_rule_fails_the_cover(monkeypatch):
    """Dropping the operand-error terms of a product (keeping only the fp32
    accumulation) leaves later tensors uncovered."""
    def acc_only(A, eA, B, eB, K):
        v = K * UA * UA * (np.abs(A) @ np.abs(B)) ** 2
        return np.sqrt(v), np.zeros(v.shape)
    monkeypatch.setattr(bounds, "matmul_err", acc_only)
    worst, _, _, _ = _worst_ratio("large-fm-sgd", seeds=(0,))
    assert max(worst.values()) > 1.0


def test_rounding_rule_second_moment_by_brute_force():
    """E[(rnd(a + D) - rnd(a))^2] <= s^2 + 6 us |a| s for D ~ N(0, s^2) and
    a spread over a rounding interval (the rule's premise)."""
    rng = np.random.default_rng(3)
    us = 2.0 ** -8
    for rel in (1e-5, 1e-3, 3e-2):
        a = rng.uniform(1.0, 2.0, 200000)
        s = rel * a
        D = rng.standard_normal(a.size) * s
        d2 = (bf16.round_bf16(a + D) - bf16.round_bf16(a)) ** 2
        assert d2.mean() <= np.mean(s * s + 6 * us * a * s)


def test_product_rule_against_fp32_accumulation():
    """fp32 matrix products of bf16 operands stay within LAMBDA s of the
    exact product (exact operands: only the accumulation term)."""
    rng = np.random.default_rng(4)
    for K in (16, 256, 2048):
        A = bf16.round_bf16(rng.standard_normal((64, K)))
        B = bf16.round_bf16(rng.standard_normal((K, 48)))
        exact = A @ B
        fp32 = (A.astype(np.float32) @ B.astype(np.float32)).astype(np.float64)
        s, m = bounds.matmul_err(A, None, B, None, K)
        assert np.all(m == 0)
        assert np.all(np.abs(fp32 - exact) <= bounds.LAMBDA * s)
