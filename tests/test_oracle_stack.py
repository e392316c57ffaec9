"""Pins for the composition of one layer of the stacked interaction
(FM block -> linear compression of vec(F) -> + residual -> LayerNorm,
Section 3.3.2 with the bias-less backbone of Section 3.3.4), and tests that
plant plausible mistakes into the oracle and check that a pin fails.

The layer is pinned through special cases whose result is known without the
oracle: with a 0/1 column-selection projection W the FM output holds Gram
entries, i.e. brute-force dot products; a 0/1 selection matrix A then places
chosen dot products at chosen output coordinates, so the vec / reshape order
is pinned; the residual is a plain matrix product C X; and LayerNorm of a
vector is (u - mean) / std with numpy's mean and population std."""
import numpy as np
import pytest

from oracle import interact
from oracle.bf16 import identity


def _brute_dot(a, b):
    s = 0.0
    for x, y in zip(a, b):
        s += float(x) * float(y)
    return s


def _ln_ref(u, gamma):
    return gamma * (u - u.mean()) / u.std()


def _selection_case(rng, n=4, d=6, n_out=3, with_C=True):
    """X, layer params with W and A 0/1 selections, plus the expected output
    computed from brute-force dot products."""
    B = 2
    X = rng.standard_normal((B, n, d))
    # W selects k = n-1 of the n Gram columns in a scrambled order:
    # W[perm[j], j] = 1, so F[i, j] = Gram[i, perm[j]] (F is not symmetric)
    k = n - 1
    perm = rng.permutation(n)[:k]
    W = np.zeros((n, k))
    W[perm, np.arange(k)] = 1.0
    # output coordinate (v, c) takes F entry (i, j) = pick[v, c]
    pick = np.stack([rng.integers(0, n, size=(n_out, d)), rng.integers(0, k, size=(n_out, d))], -1)
    A = np.zeros((n_out * d, n * k))
    for v in range(n_out):
        for c in range(d):
            i, j = pick[v, c]
            A[v * d + c, i * k + j] = 1.0       # vec_rowmajor(F)[i*k + j] = F[i, j]
    C = rng.standard_normal((n_out, n)) if with_C else np.zeros((n_out, n))
    gamma = 1.0 + 0.1 * rng.standard_normal(d)
    lay = dict(W=W, A=A, C=C, gamma=gamma)
    lay["perm"] = perm
    expect = np.zeros((B, n_out, d))
    for b in range(B):
        for v in range(n_out):
            u = np.zeros(d)
            for c in range(d):
                i, j = pick[v, c]
                u[c] = _brute_dot(X[b, i], X[b, perm[j]])
                u[c] += sum(C[v, w] * X[b, w, c] for w in range(n))
            expect[b, v] = _ln_ref(u, gamma)
    return X, lay, expect


def _maxabs(a):
    """Largest magnitude; a non-finite value counts as infinitely wrong."""
    a = np.abs(np.asarray(a, np.float64))
    return float(a.max()) if np.all(np.isfinite(a)) else float("inf")


def _run(X, layers, n_out, d, eps=0.0, fn=None):
    fn = fn or interact.stack_forward
    out, _ = fn(X, layers, n_out, d, identity, eps)
    return out


# ------------------------------------------------------------------ the pins
def check_selection(fn=None, seed=0):
    rng = np.random.default_rng(seed)
    X, lay, expect = _selection_case(rng)
    got = _run(X, [lay], 3, 6, fn=fn)
    return _maxabs(got - expect)


def check_normalised(fn=None, seed=1):
    """Each output vector divided by the gain has mean 0 and population
    variance 1 (eps = 0)."""
    rng = np.random.default_rng(seed)
    n, d, k, n_out = 5, 8, 3, 5
    X = rng.standard_normal((3, n, d))
    gamma = 1.0 + 0.2 * rng.standard_normal(d)
    lay = dict(W=rng.standard_normal((n, k)), A=rng.standard_normal((n_out * d, n * k)) * 0.1,
               C=None, gamma=gamma)
    y = _run(X, [lay], n_out, d, fn=fn) / gamma
    return max(_maxabs(y.mean(-1)), _maxabs((y ** 2).mean(-1) - 1))


def check_residual_only(fn=None, seed=2):
    """W = 0 makes the FM output, hence H, zero: the layer is LN(C X), or
    LN(X) for the identity residual."""
    rng = np.random.default_rng(seed)
    n, d, k = 4, 6, 2
    X = rng.standard_normal((2, n, d))
    gamma = 1.0 + 0.1 * rng.standard_normal(d)
    worst = 0.0
    for C, n_out in ((None, n), (rng.standard_normal((3, n)), 3)):
        lay = dict(W=np.zeros((n, k)), A=rng.standard_normal((n_out * d, n * k)), C=C, gamma=gamma)
        got = _run(X, [lay], n_out, d, fn=fn)
        for b in range(2):
            R = X[b] if C is None else C @ X[b]
            for v in range(n_out):
                worst = max(worst, _maxabs(got[b, v] - _ln_ref(R[v], gamma)))
    return worst


def check_two_layers(fn=None, seed=3):
    """A two-layer stack is the second layer applied to the first layer's
    output (each checked by the selection case)."""
    rng = np.random.default_rng(seed)
    X, lay1, e1 = _selection_case(rng, n=4, d=6, n_out=4, with_C=True)
    pick_rng = np.random.default_rng(seed + 100)
    _, lay2, _ = _selection_case(pick_rng, n=4, d=6, n_out=4, with_C=False)
    got = _run(X, [lay1, lay2], 4, 6, fn=fn)
    # second layer on the brute-force first-layer output: identity residual
    lay2b = dict(lay2, C=None)
    got2 = _run(X, [lay1, lay2b], 4, 6, fn=fn)
    exp2 = np.zeros_like(got2)
    A, g2, perm2 = lay2b["A"], lay2b["gamma"], lay2b["perm"]
    for b in range(X.shape[0]):
        Y = e1[b]
        Fm = np.array([[_brute_dot(Y[i], Y[perm2[j]]) for j in range(3)] for i in range(4)])
        H = (A @ Fm.reshape(-1)).reshape(4, 6)
        for v in range(4):
            exp2[b, v] = _ln_ref(H[v] + Y[v], g2)
    return max(_maxabs(got2 - exp2), 0.0 if np.all(np.isfinite(got)) else np.inf)


def check_lcb(fn=None, seed=4):
    """A full fusion block: the selection case's FM-block vectors followed
    by linear-compression vectors (L X, brute-force sums), then + C X and
    LayerNorm."""
    rng = np.random.default_rng(seed)
    n, d, nF, nL = 4, 6, 3, 2
    X, lay, _ = _selection_case(rng, n=n, d=d, n_out=nF, with_C=False)
    Lm = rng.standard_normal((nL, n))
    C = rng.standard_normal((nF + nL, n))
    lay = dict(lay, L=Lm, C=C)
    got = _run(X, [lay], nF + nL, d, fn=fn)
    k = n - 1
    A, perm, gamma = lay["A"], lay["perm"], lay["gamma"]
    worst = 0.0
    for b in range(X.shape[0]):
        Fm = np.array([[_brute_dot(X[b, i], X[b, perm[j]]) for j in range(k)] for i in range(n)])
        HF = (A @ Fm.reshape(-1)).reshape(nF, d)
        for v in range(nF + nL):
            u = np.zeros(d)
            for c in range(d):
                h = HF[v, c] if v < nF else sum(Lm[v - nF, w] * X[b, w, c] for w in range(n))
                u[c] = h + sum(C[v, w] * X[b, w, c] for w in range(n))
            worst = max(worst, _maxabs(got[b, v] - _ln_ref(u, gamma)))
    return worst


PINS = [check_selection, check_normalised, check_residual_only, check_two_layers, check_lcb]


@pytest.mark.parametrize("pin", PINS, ids=lambda f: f.__name__)
def test_stack_layer_pins(pin):
    assert pin() < 1e-12


# -------------------------------------------------------- planted mistakes
def _stack_variant(mistake):
    """A copy of the layer composition with one plausible mistake."""
    def fwd(X1, layers, n_out, d, rnd, eps):
        X = np.asarray(X1, np.float64)
        B = X.shape[0]
        for lay in layers:
            Fm, _ = interact.fm_forward(X, lay["W"], rnd)
            vecF = (Fm.transpose(0, 2, 1) if mistake == "vec_colmajor" else Fm).reshape(B, -1)
            nF = np.asarray(lay["A"]).shape[0] // d
            H = (vecF @ np.asarray(lay["A"]).T).reshape(B, nF, d)
            if mistake == "reshape_transposed":
                H = (vecF @ np.asarray(lay["A"]).T).reshape(B, d, nF).transpose(0, 2, 1)
            if lay.get("L") is not None:
                Lm = np.asarray(lay["L"])
                HL = np.einsum("vu,bud->bvd", Lm, X)
                if mistake == "lcb_transposed_order":
                    HL = np.einsum("vu,bud->bvd", Lm[::-1], X)
                H = np.concatenate([HL, H] if mistake == "lcb_first" else [H, HL], axis=1)
            if lay.get("C") is not None:
                R = np.einsum("vu,bud->bvd", lay["C"], X)
                if mistake == "C_transposed" and lay["C"].shape[0] == lay["C"].shape[1]:
                    R = np.einsum("uv,bud->bvd", lay["C"], X)
            else:
                R = X
            if mistake == "ln_then_residual":
                y = interact.layernorm_forward(H, lay["gamma"], eps)[0] + R
            elif mistake == "no_residual":
                y = interact.layernorm_forward(H, lay["gamma"], eps)[0]
            elif mistake == "ln_bessel":      # sample instead of population variance
                u = H + R
                y = lay["gamma"] * (u - u.mean(-1, keepdims=True)) / u.std(-1, ddof=1, keepdims=True)
            else:
                y = interact.layernorm_forward(H + R, lay["gamma"], eps)[0]
            X = rnd(y)
        return X, None
    return fwd


@pytest.mark.parametrize("mistake", ["vec_colmajor", "reshape_transposed", "ln_then_residual",
                                     "no_residual", "ln_bessel", "C_transposed", "lcb_first",
                                     "lcb_transposed_order"])
def test_planted_stack_mistakes_fail_a_pin(mistake):
    fn = _stack_variant(mistake)
    # the unmutated copy passes every pin (so a failure below is the mistake's)
    assert max(p(fn=_stack_variant(None)) for p in PINS) < 1e-12
    with np.errstate(divide="ignore", invalid="ignore"):   # LN of a zero vector in a mutated copy
        assert max(p(fn=fn) for p in PINS) > 1e-6


def test_planted_fm_mistakes_fail_a_pin():
    """FM forward with the projection applied on the wrong side, or X^T X
    instead of X X^T, fails the W = I / Gram pin of the selection case."""
    orig = interact.fm_forward

    def wrong_side(X, W, rnd):
        X = np.asarray(X, np.float64)
        P = X.transpose(0, 2, 1) @ X                     # d x d
        O = (X @ P)[:, :, :W.shape[1]]
        return O, P

    def gram_of_columns(X, W, rnd):                     # X^T X projected: d x k
        X = np.asarray(X, np.float64)
        O = (X.transpose(0, 2, 1) @ X) @ np.pad(W, ((0, max(0, X.shape[2] - W.shape[0])), (0, 0)))[:X.shape[2]]
        return O[:, :X.shape[1]], None

    for bad in (wrong_side, gram_of_columns):
        interact.fm_forward = bad
        try:
            err = check_selection()
        finally:
            interact.fm_forward = orig
        assert err > 1e-6


# ---------------------------------------------------------------------------
# FP8 projection of the FM block (Section 3.5.2: linear layers in FP8 with
# row-wise scales).  Pin: each quantised operand lies within half an e4m3
# step of its value (2^-4 relative in the normal range, 2^-10 times the
# row scale below it, plus the fp32 rounding of the scaled value), so the
# FP8 projection lies within the propagated quantisation error of the exact
# one; a projection that drops a scale, or quantises the wrong way round,
# lands far outside.

def _quant_err(x, s):
    """Bound of |dequantised - x| for row-wise e4m3 quantisation with scales s."""
    return (2.0 ** -4 + 4 * 2.0 ** -24) * np.abs(x) + 2.0 ** -10 * s[:, None]


def _fp8_case(seed=11, B=6, n=5, k=4, d=8, nv=3):
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((B, n, d)) * 0.5
    lay = dict(W=rng.standard_normal((n, k)) / np.sqrt(n),
               A=rng.standard_normal((nv * d, n * k)) / np.sqrt(n * k),
               C=rng.standard_normal((nv, n)) / np.sqrt(n), gamma=1 + 0.1 * rng.standard_normal(d))
    return X, lay, nv, d


def _projection(X, lay, nv, d, fp8):
    """(vec(F), A, H_F) of one layer: the exact projection, or the FP8 one
    written out from the quantiser and the product of the codes."""
    from oracle import fp8 as ofp8
    Fm, _ = interact.fm_forward(X, lay["W"], identity)
    vecF = Fm.reshape(X.shape[0], -1)
    A = np.asarray(lay["A"], np.float64)
    if not fp8:
        return vecF, A, vecF @ A.T
    qf, sf = ofp8.quantize(vecF)
    qa, sa = ofp8.quantize(A)
    return vecF, A, ofp8.linear_fp8(qf, sf, qa, sa)


def test_fp8_projection_within_quantisation_error():
    from oracle import fp8 as ofp8
    X, lay, nv, d = _fp8_case()
    vecF, A, exact = _projection(X, lay, nv, d, False)
    _, _, h8 = _projection(X, lay, nv, d, True)
    _, sf = ofp8.quantize(vecF)
    _, sa = ofp8.quantize(A)
    ef, ea = _quant_err(vecF, sf), _quant_err(A, sa)
    bound = ef @ np.abs(A).T + np.abs(vecF) @ ea.T + ef @ ea.T
    assert np.all(np.abs(h8 - exact) <= bound + 1e-300)
    # not vacuous: the FP8 projection does differ, by far less than its size
    assert 0 < np.max(np.abs(h8 - exact)) < 0.2 * np.max(np.abs(exact))
    # planted mistakes: a scale dropped; the weight's scales applied per
    # sample instead of per output unit
    qf, sf_ = ofp8.quantize(vecF)
    qa, sa_ = ofp8.quantize(A)
    no_scale = ofp8.linear_fp8(qf, np.ones_like(sf_), qa, sa_)
    assert np.any(np.abs(no_scale - exact) > bound)
    swapped = (ofp8.e4m3_value(qf) @ ofp8.e4m3_value(qa).T) * sf_[:, None] * sa_[:X.shape[0], None]
    assert np.any(np.abs(swapped - exact) > bound)


def test_fp8_stack_forward_uses_the_fp8_projection():
    """The stack's FP8 forward equals the bf16-free forward with its
    projection replaced by the FP8 one (checked through the LayerNorm input:
    the cached normalised values are a function of H + R alone)."""
    X, lay, nv, d = _fp8_case()
    Y8, c8 = interact.stack_forward(X, [lay], nv, d, identity, 0.0, fp8=True)
    Y, c = interact.stack_forward(X, [lay], nv, d, identity, 0.0, fp8=False)
    _, _, h8 = _projection(X, lay, nv, d, True)
    u8 = h8.reshape(X.shape[0], nv, d) + np.einsum("vu,bud->bvd", lay["C"], X)
    mu = u8.mean(axis=2, keepdims=True)
    xhat = (u8 - mu) / np.sqrt(((u8 - mu) ** 2).mean(axis=2, keepdims=True))
    np.testing.assert_allclose(c8[0]["xhat"], xhat, rtol=1e-10, atol=1e-12)
    assert not np.allclose(Y8, Y, rtol=1e-6, atol=0)      # the FP8 path was taken
    assert np.max(np.abs(Y8 - Y)) < 0.25 * np.max(np.abs(Y))
