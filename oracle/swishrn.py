"""Swish RMSNorm (SwishRN) of a feed-forward layer, its BlockNorm form and
its hard-gated variant (Sections 3.3.4 and 3.5.3).

Test infrastructure only (see the package docstring).

Definitions, for a pre-activation row ``h`` (one sample, N features) split
into normalisation groups ``G`` (``block = 0``: the whole row, i.e. RMSNorm;
``block = b``: consecutive groups of ``b`` features, the last one shorter
when ``b`` does not divide N -- BlockNorm, the statistic of one GEMM tile's
columns):

  rho_G  = 1 / sqrt(mean_{j in G} h_j^2 + eps)
  n_k    = h_k rho_G(k)                       (normalised, no gain)
  out_k  = (ga_k n_k) * gate(gb_k n_k)

with two per-feature gains: ``ga`` of the normalised value and ``gb`` of the
second RMSNorm that feeds the self-gate (reading: the gate has its own
RMSNorm, hence its own gain; both normalise the same row, so they share
``rho``).  ``gate`` is the logistic sigmoid (SwishRN) or the hard sigmoid
``clip(z / 6 + 1/2, 0, 1)`` that replaces it to avoid the exponential (with
unit gains the two forms are Swish and HardSwish of the RMS-normalised row).

Backward, from the chain rule: with ``a = ga n``, ``z = gb n``, ``s =
gate(z)`` and the output gradient ``do``:

  d ga_k = sum over samples of do_k s_k n_k
  d gb_k = sum over samples of do_k a_k gate'(z_k) n_k
  dn_k   = ga_k do_k s_k + gb_k do_k a_k gate'(z_k)
  dh_k   = rho_G (dn_k - n_k mean_{j in G}(dn_j n_j))

(``d n_k / d h_j = rho (delta_kj - n_k n_j / |G|)`` within a group, zero
across groups).  ``gate'`` of the hard sigmoid is 1/6 strictly inside
(-3, 3) and 0 outside; at the two kinks it is not defined and either
one-sided value is a correct result.
"""
import numpy as np

GATES = ("sigmoid", "hard")


def gate(z, kind):
    z = np.asarray(z, np.float64)
    if kind == "sigmoid":
        return 0.5 * (1.0 + np.tanh(0.5 * z))    # = 1 / (1 + exp(-z)), no overflow
    if kind == "hard":
        return np.clip(z / 6.0 + 0.5, 0.0, 1.0)
    raise ValueError(kind)


def gate_grad(z, kind):
    z = np.asarray(z, np.float64)
    if kind == "sigmoid":
        s = gate(z, kind)
        return s * (1.0 - s)
    if kind == "hard":
        return np.where(np.abs(z) < 3.0, 1.0 / 6.0, 0.0)
    raise ValueError(kind)


def groups(N, block):
    """Column ranges ``[(lo, hi), ...]`` of the normalisation groups."""
    if block <= 0 or block >= N:
        return [(0, N)]
    return [(lo, min(lo + block, N)) for lo in range(0, N, block)]


def rms_inv(h, block, eps):
    """``rho`` of every row and group: ``[M, n_groups]``."""
    h = np.asarray(h, np.float64)
    return np.stack([1.0 / np.sqrt(np.mean(h[:, lo:hi] ** 2, axis=1) + eps)
                     for lo, hi in groups(h.shape[1], block)], axis=1)


def expand(rho, N, block):
    """Per-group values ``[M, n_groups]`` broadcast to their columns ``[M, N]``."""
    out = np.empty((rho.shape[0], N))
    for g, (lo, hi) in enumerate(groups(N, block)):
        out[:, lo:hi] = rho[:, g:g + 1]
    return out


def forward(h, ga, gb, block, eps, kind, rho=None):
    """Returns ``(out, n, rho)``.  ``rho`` (optional) replaces the statistic
    computed from ``h`` (the backward of an accelerator that stored it)."""
    h = np.asarray(h, np.float64)
    ga, gb = np.asarray(ga, np.float64), np.asarray(gb, np.float64)
    rho = rms_inv(h, block, eps) if rho is None else np.asarray(rho, np.float64)
    n = h * expand(rho, h.shape[1], block)
    return ga * n * gate(gb * n, kind), n, rho


def backward(do, h, ga, gb, block, eps, kind, rho=None, grad_override=None):
    """Returns ``(dh, dga, dgb)`` given ``do = dL/d out``.
    ``grad_override`` (optional, hard gate): ``(where, value)``, the value
    ``gate'`` takes at the positions ``where`` instead of its own (parity
    tests use it only where the side of a kink at +-3 is not fixed by the
    arithmetic; either one-sided derivative is then a correct result)."""
    do = np.asarray(do, np.float64)
    ga, gb = np.asarray(ga, np.float64), np.asarray(gb, np.float64)
    _, n, rho = forward(h, ga, gb, block, eps, kind, rho)
    a, z = ga * n, gb * n
    s, sp = gate(z, kind), gate_grad(z, kind)
    if grad_override is not None:
        where, value = grad_override
        sp = np.where(where, value, sp)
    da = do * s
    dz = do * a * sp
    dga = (da * n).sum(axis=0)
    dgb = (dz * n).sum(axis=0)
    dn = ga * da + gb * dz
    N = n.shape[1]
    dh = np.empty_like(dn)
    for g, (lo, hi) in enumerate(groups(N, block)):
        m = np.mean(dn[:, lo:hi] * n[:, lo:hi], axis=1, keepdims=True)
        dh[:, lo:hi] = rho[:, g:g + 1] * (dn[:, lo:hi] - n[:, lo:hi] * m)
    return dh, dga, dgb


# --- how far a correct fp32 evaluation may lie from the float64 value -------

U32 = 2.0 ** -24
_GP = {"sigmoid": 0.25, "hard": 1.0 / 6.0}     # max |gate'|
_GPP = {"sigmoid": 0.1, "hard": 0.0}          # max |gate''| (1 / (6 sqrt 3) < 0.1)


def forward_bound(h, eh, ga, gb, block, eps, kind):
    """Element-wise bounds ``(e_out, e_rho)`` on the difference between an
    fp32 evaluation of ``forward`` and the float64 one, when the
    accelerator's pre-activation differs from ``h`` by at most ``eh`` (its
    GEMM's accumulation error; 0 when it normalises the stored ``h``
    itself), to first order with a factor 1.25 for the rest:

    * ``|d n_k| <= rho eh_k + |n_k| rho^2 sum_G |h_j| eh_j / |G|`` plus the
      fp32 evaluation of ``rho`` (a sum of |G| squares, a reciprocal square
      root and the product: ``(|G|/2 + 5) 2^-24`` relative);
    * ``out`` moves by at most ``L |d n|`` with the derivative bound ``L =
      |ga| (gate(z) + |gb| |d n| max|gate'| + (|z| + |gb| |d n|) max|gate'|)``
      over the interval, plus 8 fp32 roundings of ``|out| + |ga n|`` (the
      gate's exponential and reciprocal, the products)."""
    h = np.asarray(h, np.float64)
    eh = np.broadcast_to(np.asarray(eh, np.float64), h.shape)
    ga, gb = np.asarray(ga, np.float64), np.asarray(gb, np.float64)
    out, n, rho = forward(h, ga, gb, block, eps, kind)
    N = h.shape[1]
    R = expand(rho, N, block)
    sz = np.empty_like(h)
    gsize = np.empty_like(h)
    for lo, hi in groups(N, block):
        sz[:, lo:hi] = np.sum(np.abs(h[:, lo:hi]) * eh[:, lo:hi], axis=1, keepdims=True) / (hi - lo)
        gsize[:, lo:hi] = hi - lo
    en = R * eh + np.abs(n) * R * R * sz + np.abs(n) * (gsize / 2 + 5) * U32
    z = gb * n
    gp = _GP[kind]
    L = np.abs(ga) * (np.minimum(1.0, gate(z, kind) + np.abs(gb) * en * gp) + (np.abs(z) + np.abs(gb) * en) * gp)
    e_out = 1.25 * (L * en + 8 * U32 * (np.abs(out) + np.abs(ga * n)))
    gs = np.array([hi - lo for lo, hi in groups(N, block)], np.float64)
    e_rho = 1.25 * (rho ** 3 * _group_mean(np.abs(h) * eh, block) + rho * (gs / 2 + 5) * U32)
    return e_out, e_rho


def _group_mean(x, block):
    return np.stack([np.mean(x[:, lo:hi], axis=1) for lo, hi in groups(x.shape[1], block)], axis=1)


def backward_bound(do, edo, h, ga, gb, block, eps, kind, rho, n_rows_summed=None):
    """Element-wise bounds ``(e_dh, e_dga, e_dgb)`` on an fp32 evaluation of
    ``backward`` from the stored ``h`` and ``rho`` when the accelerator's
    output gradient differs from ``do`` by at most ``edo``.  ``dh`` is linear
    in ``do`` with coefficients ``c = ga s + gb a gate'``:

      |d dh_j| <= rho (|c_j| edo_j + |n_j| sum_G |c_k n_k| edo_k / |G|)

    plus fp32 evaluation errors: 12 roundings on ``c`` (relative to ``cabs
    = |ga|(s + |z| max|gate'|) + |gb a|(gate' + |z| max|gate''|)``), one on
    ``dn``, ``|G| + 2`` in the group mean, three in the final expression.
    At a kink of the hard gate (``|z|`` within 2^-20 relative of 3) ``dn``
    may also jump by ``|do gb a| / 6``.  The gain gradients sum ``B`` rows:
    the propagated error plus ``B + 12`` roundings of the absolute sum."""
    do = np.asarray(do, np.float64)
    edo = np.broadcast_to(np.asarray(edo, np.float64), do.shape)
    ga, gb = np.asarray(ga, np.float64), np.asarray(gb, np.float64)
    _, n, rho = forward(h, ga, gb, block, eps, kind, rho)
    N = n.shape[1]
    R = expand(rho, N, block)
    a, z = ga * n, gb * n
    s, sp = gate(z, kind), gate_grad(z, kind)
    gp, gpp = _GP[kind], _GPP[kind]
    c = ga * s + gb * a * sp
    cabs = np.abs(ga) * (s + np.abs(z) * gp) + np.abs(gb * a) * (sp + np.abs(z) * gpp)
    jump = np.zeros_like(n)
    if kind == "hard":
        amb = np.abs(np.abs(z) - 3.0) <= 2.0 ** -20 * 3.0
        jump = np.where(amb, np.abs(do * gb * a) / 6.0, 0.0)
    dn = c * do
    e_dn = np.abs(c) * edo + 12 * U32 * cabs * np.abs(do) + U32 * np.abs(dn) + jump
    spread = np.empty_like(n)
    mabs = np.empty_like(n)
    for lo, hi in groups(N, block):
        G = hi - lo
        spread[:, lo:hi] = (np.sum(e_dn[:, lo:hi] * np.abs(n[:, lo:hi]), axis=1, keepdims=True) / G
                            + (G + 2) * U32 * np.sum(np.abs(dn[:, lo:hi] * n[:, lo:hi]), axis=1, keepdims=True) / G)
        mabs[:, lo:hi] = np.abs(np.mean(dn[:, lo:hi] * n[:, lo:hi], axis=1, keepdims=True))
    e_dh = 1.25 * R * (e_dn + np.abs(n) * spread + 3 * U32 * (np.abs(dn) + np.abs(n) * mabs))
    B = do.shape[0] if n_rows_summed is None else n_rows_summed
    e_dga = 1.25 * ((np.abs(s * n) * edo + 12 * U32 * np.abs(do * n) * (s + np.abs(z) * gp)).sum(0)
                    + (B + 12) * U32 * np.abs(do * s * n).sum(0))
    dz_abs = np.abs(do * a * n)
    e_dgb = 1.25 * ((np.abs(a * sp * n) * edo + 12 * U32 * dz_abs * (sp + np.abs(z) * gpp) + jump * np.abs(n)).sum(0)
                    + (B + 12) * U32 * (dz_abs * sp).sum(0))
    return e_dh, e_dga, e_dgb
