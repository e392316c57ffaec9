"""Pins of the oracle's SwishRN / BlockNorm / hard-gate layer (Sections 3.3.4
and 3.5.3) against what is fixed independently of it: torch's own RMSNorm,
SiLU, HardSwish and hard-sigmoid routines (float64, CPU), the invariances of
a normalisation, closed forms at special gains, torch's autograd of the
library composition, and the error bounds against perturbed evaluations."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import swishrn

RNG = np.random.default_rng(2512)


def _rows(M, N, scale=1.0):
    return RNG.standard_normal((M, N)) * scale


def _t(x):
    return torch.from_numpy(np.asarray(x, np.float64))


def _lib(h, ga, gb, block, eps, kind):
    """The definition from torch's routines, group by group."""
    N = h.shape[1]
    out = torch.empty(h.shape, dtype=torch.float64)
    gate = torch.sigmoid if kind == "sigmoid" else F.hardsigmoid
    for lo, hi in ([(0, N)] if block == 0 else [(lo, min(lo + block, N)) for lo in range(0, N, block)]):
        x = _t(h[:, lo:hi])
        a = F.rms_norm(x, (hi - lo,), _t(ga[lo:hi]), eps)
        z = F.rms_norm(x, (hi - lo,), _t(gb[lo:hi]), eps)
        out[:, lo:hi] = a * gate(z)
    return out.numpy()


@pytest.mark.parametrize("kind", swishrn.GATES)
def test_unit_gains_are_swish_and_hardswish_of_rmsnorm(kind):
    h = _rows(9, 37, 3.0)
    one = np.ones(37)
    out, _, _ = swishrn.forward(h, one, one, 0, 1e-6, kind)
    x = F.rms_norm(_t(h), (37,), eps=1e-6)
    ref = (F.silu(x) if kind == "sigmoid" else F.hardswish(x)).numpy()
    assert np.max(np.abs(out - ref)) < 1e-13


@pytest.mark.parametrize("kind", swishrn.GATES)
@pytest.mark.parametrize("N,block", [(64, 0), (200, 64), (200, 128), (130, 128), (96, 200)])
def test_two_gains_and_blocknorm_groups_match_the_library(kind, N, block):
    h = _rows(11, N, 2.0)
    ga, gb = 1 + 0.3 * RNG.standard_normal(N), 1 + 0.3 * RNG.standard_normal(N)
    out, n, rho = swishrn.forward(h, ga, gb, block, 1e-5, kind)
    assert np.max(np.abs(out - _lib(h, ga, gb, block, 1e-5, kind))) < 1e-13
    G = swishrn.groups(N, block)
    assert rho.shape == (11, len(G))
    assert G[-1][1] == N and all(hi - lo == (block if block and block < N else N) for lo, hi in G[:-1])


def test_blocknorm_scale_invariance_per_group_rmsnorm_per_row():
    """eps = 0: scaling every group by its own positive factor leaves
    BlockNorm unchanged but not the whole-row RMSNorm; scaling the whole row
    leaves both unchanged; each group of n has mean square 1."""
    N, b = 256, 128
    h = _rows(5, N)
    ga, gb = 1 + 0.2 * RNG.standard_normal(N), 1 + 0.2 * RNG.standard_normal(N)
    c = np.concatenate([np.full(b, 3.0), np.full(b, 0.25)])
    for kind in swishrn.GATES:
        blk, n, _ = swishrn.forward(h, ga, gb, b, 0.0, kind)
        assert np.max(np.abs(swishrn.forward(h * c, ga, gb, b, 0.0, kind)[0] - blk)) < 1e-13
        row, _, _ = swishrn.forward(h, ga, gb, 0, 0.0, kind)
        assert np.max(np.abs(swishrn.forward(h * c, ga, gb, 0, 0.0, kind)[0] - row)) > 1e-2
        assert np.max(np.abs(swishrn.forward(h * 7.5, ga, gb, 0, 0.0, kind)[0] - row)) < 1e-13
        for lo, hi in swishrn.groups(N, b):
            assert np.allclose(np.mean(n[:, lo:hi] ** 2, axis=1), 1.0, rtol=0, atol=1e-13)


@pytest.mark.parametrize("kind", swishrn.GATES)
def test_special_gains(kind):
    """ga = 0 gives zero; gb = 0 opens every gate half way (sigmoid(0) =
    hard-sigmoid(0) = 1/2): half the gained RMSNorm."""
    N = 48
    h = _rows(6, N)
    ga = 1 + 0.3 * RNG.standard_normal(N)
    out, _, _ = swishrn.forward(h, np.zeros(N), ga, 16, 1e-6, kind)
    assert np.all(out == 0)
    out, _, _ = swishrn.forward(h, ga, np.zeros(N), 16, 1e-6, kind)
    ref = np.concatenate([F.rms_norm(_t(h[:, lo:lo + 16]), (16,), _t(ga[lo:lo + 16]), 1e-6).numpy()
                          for lo in range(0, N, 16)], axis=1)
    assert np.max(np.abs(out - 0.5 * ref)) < 1e-13


def test_hard_gate_saturates_and_has_no_exponential_tail():
    z = np.array([-9.0, -3.0, -1.5, 0.0, 1.5, 3.0, 9.0])
    assert np.array_equal(swishrn.gate(z, "hard"), [0.0, 0.0, 0.25, 0.5, 0.75, 1.0, 1.0])
    assert np.array_equal(swishrn.gate_grad(z, "hard"), [0, 0, 1 / 6, 1 / 6, 1 / 6, 0, 0])


@pytest.mark.parametrize("kind", swishrn.GATES)
@pytest.mark.parametrize("N,block", [(40, 0), (70, 32), (128, 128)])
def test_backward_matches_autograd_of_the_library_composition(kind, N, block):
    M = 13
    h = _rows(M, N, 1.5)
    ga, gb = 1 + 0.3 * RNG.standard_normal(N), 1 + 0.3 * RNG.standard_normal(N)
    do = RNG.standard_normal((M, N))
    if kind == "hard":
        _, n, _ = swishrn.forward(h, ga, gb, block, 1e-4, kind)
        assert np.min(np.abs(np.abs(gb * n) - 3)) > 1e-6
    th, tga, tgb = (_t(x).requires_grad_() for x in (h, ga, gb))
    # (torch's float64 hard-sigmoid backward scales by 1/6 rounded to fp32,
    # a 3e-8 relative error, so the hard gate is written out with clamp)
    gate = torch.sigmoid if kind == "sigmoid" else (lambda z: torch.clamp(z / 6 + 0.5, 0.0, 1.0))
    parts = []
    for lo, hi in ([(0, N)] if block == 0 else [(lo, min(lo + block, N)) for lo in range(0, N, block)]):
        x = th[:, lo:hi]
        parts.append(F.rms_norm(x, (hi - lo,), tga[lo:hi], 1e-4) * gate(F.rms_norm(x, (hi - lo,), tgb[lo:hi], 1e-4)))
    (torch.cat(parts, dim=1) * _t(do)).sum().backward()
    dh, dga, dgb = swishrn.backward(do, h, ga, gb, block, 1e-4, kind)
    for got, ref in ((dh, th.grad), (dga, tga.grad), (dgb, tgb.grad)):
        ref = ref.numpy()
        assert np.max(np.abs(got - ref)) <= 1e-11 * max(1.0, np.max(np.abs(ref)))


@pytest.mark.parametrize("kind", swishrn.GATES)
def test_backward_central_differences(kind):
    M, N, block = 4, 20, 8
    h = _rows(M, N)
    ga, gb = 1 + 0.3 * RNG.standard_normal(N), 1 + 0.3 * RNG.standard_normal(N)
    w = RNG.standard_normal((M, N))
    dh, dga, dgb = swishrn.backward(w, h, ga, gb, block, 1e-3, kind)

    def L():
        return float(np.sum(w * swishrn.forward(h, ga, gb, block, 1e-3, kind)[0]))
    for arr, grad in ((h, dh), (ga, dga), (gb, dgb)):
        for idx in np.ndindex(arr.shape):
            old = arr[idx]
            arr[idx] = old + 1e-6
            lp = L()
            arr[idx] = old - 1e-6
            lm = L()
            arr[idx] = old
            assert abs((lp - lm) / 2e-6 - grad[idx]) < 1e-6 * max(1.0, np.max(np.abs(grad)))


@pytest.mark.parametrize("kind", swishrn.GATES)
@pytest.mark.parametrize("block", [0, 128])
def test_bounds_cover_perturbed_evaluations(kind, block):
    """The forward bound covers the oracle's own value at pre-activations
    moved anywhere inside ``eh`` (sign patterns at the corners, where a
    first-order bound is tightest), and is not vacuous; the backward bound
    likewise for output gradients moved inside ``edo``."""
    M, N = 64, 200
    h = _rows(M, N)
    ga, gb = 1 + 0.3 * RNG.standard_normal(N), 1 + 0.3 * RNG.standard_normal(N)
    eh = 1e-4 * (np.abs(h) + 0.5)
    out, _, rho = swishrn.forward(h, ga, gb, block, 1e-6, kind)
    e_out, e_rho = swishrn.forward_bound(h, eh, ga, gb, block, 1e-6, kind)
    worst = 0.0
    for trial in range(20):
        sgn = RNG.choice([-1.0, 1.0], size=h.shape)
        o2, _, r2 = swishrn.forward(h + sgn * eh, ga, gb, block, 1e-6, kind)
        worst = max(worst, np.max(np.abs(o2 - out) / e_out))
        assert np.all(np.abs(r2 - rho) <= e_rho)
    assert 0.05 < worst <= 1.0, worst
    do = RNG.standard_normal((M, N))
    edo = 1e-4 * (np.abs(do) + 0.1)
    dh, dga, dgb = swishrn.backward(do, h, ga, gb, block, 1e-6, kind, rho)
    e_dh, e_dga, e_dgb = swishrn.backward_bound(do, edo, h, ga, gb, block, 1e-6, kind, rho)
    worst = 0.0
    for trial in range(20):
        sgn = RNG.choice([-1.0, 1.0], size=h.shape)
        d2 = swishrn.backward(do + sgn * edo, h, ga, gb, block, 1e-6, kind, rho)
        worst = max(worst, max(float(np.max(np.abs(x - y) / e)) for x, y, e in
                               zip(d2, (dh, dga, dgb), (e_dh, e_dga, e_dgb))))
    assert 0.05 < worst <= 1.0, worst


def test_gate_derivative_override_is_local_to_its_group():
    """Overriding the hard gate's derivative with its own value changes
    nothing; changing it at one element changes dh only inside that
    element's normalisation group, and the gain gradients only in its
    column."""
    M, N, block = 6, 40, 16
    h = _rows(M, N, 2.0)
    ga, gb = 1 + 0.3 * RNG.standard_normal(N), 1 + 0.3 * RNG.standard_normal(N)
    do = RNG.standard_normal((M, N))
    _, n, _ = swishrn.forward(h, ga, gb, block, 1e-6, "hard")
    z = gb * n
    base = swishrn.backward(do, h, ga, gb, block, 1e-6, "hard")
    same = swishrn.backward(do, h, ga, gb, block, 1e-6, "hard",
                            grad_override=(np.ones((M, N), bool), swishrn.gate_grad(z, "hard")))
    for a, b in zip(base, same):
        assert np.array_equal(a, b)
    r, k = 2, 21                                  # group 1 (columns 16..31)
    where = np.zeros((M, N), bool)
    where[r, k] = True
    val = np.full((M, N), 1 / 6 - swishrn.gate_grad(z, "hard")[r, k])   # flip 0 <-> 1/6
    dh, dga, dgb = swishrn.backward(do, h, ga, gb, block, 1e-6, "hard", grad_override=(where, val))
    changed = dh != base[0]
    assert changed[r, 16:32].any() and not changed[:, :16].any() and not changed[:, 32:].any()
    assert not changed[np.arange(M) != r].any()
    assert np.array_equal(dga, base[1])
    assert np.flatnonzero(dgb != base[2]).tolist() == [k]
