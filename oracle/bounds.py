"""Element-wise error scales for comparing an accelerator's training step
with the oracle: how far apart two correct evaluations of the step may lie.

Test infrastructure only (see the package docstring).

Both sides evaluate the same definition on the same inputs; they differ only
in arithmetic.  The accelerator accumulates products in fp32 (unit roundoff
``UA = 2^-24``; bf16 x bf16 products are exact in fp32) in an order of its
own, and both sides round every stored tensor to the storage grid (unit
roundoff ``us = 2^-8`` for bfloat16, ``2^-24`` for fp32 storage).

Worst-case bounds (every rounding error taken with the same sign) grow by
about sqrt(K) per contraction of K terms and say nothing after a few layers.
Rounding errors behave as independent zero-mean variables instead (the
probabilistic rounding-error analysis of Higham and Mary, SIAM J. Sci.
Comput. 41(5), 2019).  But a stored value differs between the two sides only
when their small accumulation differences carry it across a rounding
boundary: a rare jump of one ulp, not a small Gaussian error.  So every
stored tensor ``Y`` of the oracle's step carries two element-wise scales of
``Y_acc - Y_oracle``, propagated to first order through the same sequence of
operations, with errors of distinct elements independent:

* ``s``: a bound on the standard deviation (second moment) of the
  difference;
* ``m``: a bound on the largest single jump, i.e. the effect of one rounding
  flip of one operand element, that can reach the element.

Rules:

* a product ``Y = A B`` over ``K`` terms, accumulated in fp32 in any order:
  ``s_Y^2 = A^2 s_B^2 + s_A^2 B^2 + K UA^2 (|A| |B|)^2`` and
  ``m_Y = max_k |A_ik| * max_k m_B,kj + max_k m_A,ik * max_k |B_kj|``;
* a value both sides round to the storage grid (ulp <= 2 us |y|): a
  difference ``D`` before rounding becomes ``D'`` with ``|D' - D| <= ulp``,
  and ``D' != D`` only where D carries the value across a rounding
  boundary, so ``E[D'^2] <= E[D^2] + 3 ulp E|D|``: ``s^2 <- s^2 + 6 us |y| s``
  and ``m <- max(m (1 + us), 2 us |y|)``;
* ReLU is 1-Lipschitz and passes both through; in the backward pass a ReLU
  decision is ambiguous where the oracle's pre-activation lies within the
  accepted deviation of zero, and there the masked gradient may differ by
  the whole unmasked value (a jump);
* LayerNorm, the sigmoid of the loss and the transcendental functions add
  their linearised sensitivities and a few fp32 roundings.

A parity test accepts an element when ``|x - r| <= LAMBDA s + JUMPS m``: the
many-source part within ``LAMBDA = 8`` standard deviations (a normal tail of
1e-15 per element) plus up to ``JUMPS = 3`` maximal single jumps (where
flips are common, a few of them can reach one element together with nearly
their largest effect; the second moment ``s`` already counts them, but not
their heavy tail).
``step_bounds`` mirrors ``step.forward`` and ``step.backward`` and returns
``(s, m)`` for every tensor the parity tests compare, keyed like the oracle's
outputs; ``allowed`` turns a pair into the accepted deviation.
"""
import numpy as np

from .embbag import pool_forward, pool_backward, row_keys
from .interact import pair_indices, fm_backward, dot_backward
from .loss import sigmoid

UA = 2.0 ** -24
LAMBDA = 8.0
JUMPS = 3.0


def storage_unit(dtype):
    return 2.0 ** -8 if dtype == "bf16" else 2.0 ** -24


def allowed(e):
    """Accepted |accelerator - oracle| of each element given its (s, m)."""
    s, m = e
    return LAMBDA * s + JUMPS * m


def _sq(x):
    return x * x


def rounded(e, y, us):
    """(s, m) after both sides round to the storage grid."""
    s, m = e
    ay = np.abs(y)
    return np.sqrt(_sq(s) + 6.0 * us * ay * s), np.maximum(m * (1.0 + us), 2.0 * us * ay)


def _rowmax(x):
    return np.abs(x).max(axis=-1, keepdims=True) if x.shape[-1] else np.zeros(x.shape[:-1] + (1,))


def _colmax(x):
    return (np.abs(x).max(axis=-2, keepdims=True) if x.shape[-2]
            else np.zeros(x.shape[:-2] + (1,) + x.shape[-1:]))


def matmul_err(A, eA, B, eB, K):
    """(s, m) of ``A @ B`` (batched allowed) given those of A and B
    (``None``: exact operand), accumulated over K terms in fp32."""
    v = K * UA * UA * _sq(np.abs(A) @ np.abs(B))
    m = np.zeros(v.shape)
    if eB is not None:
        v = v + _sq(A) @ _sq(eB[0])
        m = m + _rowmax(A) * _colmax(eB[1])
    if eA is not None:
        v = v + _sq(eA[0]) @ _sq(B)
        m = m + _rowmax(eA[1]) * _colmax(B)
    return np.sqrt(v), m


def _add(*es):
    """(s, m) of a sum of independent differences."""
    return np.sqrt(sum(_sq(e[0]) for e in es)), sum(e[1] for e in es)


def _T(x):
    return x.transpose(0, 2, 1)


def _Te(e):
    return _T(e[0]), _T(e[1])


def _Te2(e):
    return e[0].T, e[1].T


def _scale(e, c):
    c = np.abs(c)
    return e[0] * c, e[1] * c


def _mlp_forward_bounds(hs, layers, eh0, us, last_linear):
    """(s, m) of every layer output and, per layer, the pre-activation with
    its (s, m), of a forward MLP."""
    eh = [eh0]
    pre = []
    for i, (W, b) in enumerate(layers):
        W = np.asarray(W, np.float64)
        b = np.asarray(b, np.float64)
        a = hs[i] @ W.T + b
        s = np.sqrt((W.shape[1] + 3) * UA * UA) * (np.abs(hs[i]) @ np.abs(W).T + np.abs(b))
        ea = (s, np.zeros(s.shape))
        if eh[-1] is not None:
            ea = _add(ea, matmul_err(hs[i], eh[-1], W.T, None, 0))
        pre.append((a, ea))
        if last_linear and i == len(layers) - 1:
            eh.append(_add(ea, (UA * np.abs(a), 0.0)))
        else:
            eh.append(rounded(ea, hs[i + 1], us))
    return eh, pre


def _masked(dh, edh, mask, a, ea):
    """(s, m) of the ReLU-masked gradient: where the decision is ambiguous
    the two sides may differ by the whole unmasked value."""
    amb = np.abs(a) <= allowed(ea)
    s = np.where(mask, edh[0], 0.0)
    m = np.where(amb, np.abs(dh) + allowed(edh), np.where(mask, edh[1], 0.0))
    return s, m


def _mlp_backward_bounds(g, eg, hs, eh, masks, pre, layers, rnd, us, need_input):
    """(s, m) of dW, db of every layer (and of the input gradient) given the
    stored gradient ``g`` of the last layer's output."""
    L = len(layers)
    B = g.shape[0]
    dW, db = [None] * L, [None] * L
    e_in, g_in = None, None
    for i in range(L - 1, -1, -1):
        W = np.asarray(layers[i][0], np.float64)
        dW[i] = matmul_err(g.T, _Te2(eg), hs[i], eh[i], B)
        db[i] = (np.sqrt(_sq(eg[0]).sum(0) + B * UA * UA * _sq(np.abs(g).sum(0))),
                 eg[1].max(0) if B else np.zeros(g.shape[1]))
        if i == 0 and not need_input:
            break
        dh = g @ W
        edh = matmul_err(g, eg, W, None, W.shape[0])
        if i > 0:
            a, ea = pre[i - 1]
            e = _masked(dh, edh, masks[i - 1], a, ea)
            g = rnd(dh * masks[i - 1])
            eg = rounded(e, g, us)
        else:
            g_in, e_in = dh, edh
    return dW, db, g_in, e_in


def _layernorm_forward_bounds(u, eu, xhat, rstd):
    """(s, m) of x-hat and of rstd given those of the LayerNorm input
    (linearised), plus the fp32 evaluation of mean, variance and the
    normalisation."""
    d = u.shape[-1]
    mn = lambda x: x.mean(-1, keepdims=True)
    mx = lambda x: x.max(-1, keepdims=True)
    dev = u - mn(u)
    var_eps = 1.0 / rstd ** 2                 # variance + eps
    err_mu = (d + 2) * UA * mn(np.abs(u))
    rel_rstd = ((d + 4) * UA * mn(dev ** 2) + 2 * mn(np.abs(dev)) * err_mu) / (2 * var_eps) + 3 * UA
    v, m = _sq(eu[0]), eu[1]
    ax = np.abs(xhat)
    s_r = np.sqrt(_sq(rstd ** 2) * mn(_sq(xhat) * v) / d + _sq(rstd * rel_rstd))
    m_r = rstd ** 2 * mx(ax * m) / d
    s_x = np.sqrt(_sq(rstd) * (v + mn(v) / d + _sq(xhat) * mn(_sq(xhat) * v) / d)
                  + _sq(rstd * err_mu + ax * (rel_rstd + 2 * UA)))
    m_x = rstd * (m + mx(m) * (1 + ax * mx(ax)) / d)
    return (s_x, m_x), (s_r, m_r)


def _fm_forward_bounds(X, eX, W, P, O, us):
    n, d = X.shape[1], X.shape[2]
    eP = rounded(matmul_err(_T(X), _Te(eX), W, None, n), P, us)
    eO = rounded(matmul_err(X, eX, P, eP, d), O, us)
    return eP, eO


def _fm_backward_bounds(G, eG, X, eX, W, P, eP, rnd, us):
    """(s, m) of dX (unrounded sum) and dW of the FM block."""
    B, n, d = X.shape
    k = W.shape[1]
    dP = rnd(_T(X) @ G)
    edP = rounded(matmul_err(_T(X), _Te(eX), G, eG, n), dP, us)
    Wb = np.broadcast_to(W[None], (B,) + W.shape)
    edX = _add(matmul_err(G, eG, _T(P), _Te(eP), k), matmul_err(Wb, None, _T(dP), _Te(edP), k))
    # dW = sum_b X_b dP_b: the per-sample products' differences add over b
    sb, mb = _add(matmul_err(X, eX, dP, None, 0), matmul_err(X, None, dP, edP, 0))
    sdW = np.sqrt(_sq(sb).sum(0) + B * d * UA * UA * _sq((np.abs(X) @ np.abs(dP)).sum(0)))
    return edX, (sdW, mb.max(0))


def _stack_forward_bounds(layers, caches, eX, d, rnd, us):
    """(s, m) of the stacked interaction's output, and per layer the scales
    its backward needs."""
    mean = lambda x: x.mean(-1, keepdims=True)
    B = eX[0].shape[0]
    st_fwd = []
    eXl = eX
    for lay, cl in zip(layers, caches):
        Xl, P = cl["X"], cl["P"]
        nl = Xl.shape[1]
        W = np.asarray(lay["W"], np.float64)
        k = W.shape[1]
        vecF = cl["vecF"]
        ePl, eF = _fm_forward_bounds(Xl, eXl, W, P, vecF.reshape(B, nl, k), us)
        eF2 = (eF[0].reshape(B, -1), eF[1].reshape(B, -1))
        A = np.asarray(lay["A"], np.float64)
        eH = matmul_err(vecF, eF2, A.T, None, nl * k)
        eH = (eH[0].reshape(B, -1, d), eH[1].reshape(B, -1, d))
        H = (vecF @ A.T).reshape(B, -1, d)
        if lay.get("L") is not None:              # linear compression block rows
            Lm = np.asarray(lay["L"], np.float64)
            Lb = np.broadcast_to(Lm[None], (B,) + Lm.shape)
            eHL = matmul_err(Lb, None, Xl, eXl, nl)
            H = np.concatenate([H, Lb @ Xl], axis=1)
            eH = (np.concatenate([eH[0], eHL[0]], axis=1), np.concatenate([eH[1], eHL[1]], axis=1))
        if lay.get("C") is not None:
            C = np.asarray(lay["C"], np.float64)
            Cb = np.broadcast_to(C[None], (B,) + C.shape)
            R = Cb @ Xl
            eR = matmul_err(Cb, None, Xl, eXl, nl)
        else:
            R, eR = Xl, eXl
        u = H + R
        eu = _add(eH, eR, (UA * np.abs(u), 0.0))
        ex, er = _layernorm_forward_bounds(u, eu, cl["xhat"], cl["rstd"])
        gam = np.asarray(lay["gamma"], np.float64)
        y = gam * cl["xhat"]
        st_fwd.append(dict(eX=eXl, eP=ePl, eF=eF, ex=ex, er=er))
        eXl = rounded(_add(_scale(ex, gam), (UA * np.abs(y), 0.0)), rnd(y), us)
    return eXl, st_fwd


def _stack_backward_bounds(layers, caches, st_fwd, dY, edY, rnd, us):
    """(s, m) of the stacked interaction's input gradient and of every
    layer's parameter gradients, given the stored output gradient dY."""
    mean = lambda x: x.mean(-1, keepdims=True)
    mx = lambda x: x.max(-1, keepdims=True)
    B, nv, d = dY.shape
    grads = [None] * len(layers)
    for li in range(len(layers) - 1, -1, -1):
        lay, cl, sf = layers[li], caches[li], st_fwd[li]
        Xl, P, xhat, rstd = cl["X"], cl["P"], cl["xhat"], cl["rstd"]
        nl = Xl.shape[1]
        gam = np.asarray(lay["gamma"], np.float64)
        W = np.asarray(lay["W"], np.float64)
        k = W.shape[1]
        A = np.asarray(lay["A"], np.float64)
        ax = np.abs(xhat)
        dxh = dY * gam
        edxh = _scale(edY, gam)
        s1 = mean(dxh * xhat)
        du = rstd * (dxh - mean(dxh) - xhat * s1)
        vdxh, vx = _sq(edxh[0]), _sq(sf["ex"][0])
        sdu = np.sqrt(_sq(rstd) * (vdxh + mean(vdxh) / d
                                   + _sq(xhat) * mean(_sq(xhat) * vdxh + _sq(dxh) * vx) / d + vx * _sq(s1))
                      + _sq(sf["er"][0] * du / rstd)
                      + _sq((2 * d + 8) * UA * rstd * (np.abs(dxh) + mean(np.abs(dxh)))))
        mdu = (rstd * (edxh[1] + mx(edxh[1]) * (1 + ax * mx(ax)) / d + sf["ex"][1] * np.abs(s1)
                       + ax * mx(np.abs(dxh) * sf["ex"][1]) / d)
               + sf["er"][1] * np.abs(du) / rstd)
        edu = (sdu, mdu)
        edg = (np.sqrt((_sq(edY[0] * xhat) + _sq(dY) * vx).reshape(-1, d).sum(0)
                       + B * nv * UA * UA * _sq(np.abs(dY * xhat).reshape(-1, d).sum(0))),
               (edY[1] * ax + np.abs(dY) * sf["ex"][1]).reshape(-1, d).max(0))
        duR = rnd(du)
        eduR = rounded(edu, duR, us)
        nF = A.shape[0] // d
        du2 = duR[:, :nF].reshape(B, -1)
        edu2 = (eduR[0][:, :nF].reshape(B, -1), eduR[1][:, :nF].reshape(B, -1))
        vecF = cl["vecF"]
        eF2 = (sf["eF"][0].reshape(B, -1), sf["eF"][1].reshape(B, -1))
        edA = matmul_err(du2.T, _Te2(edu2), vecF, eF2, B)
        dF = rnd((du2 @ A).reshape(B, nl, k))
        edF = matmul_err(du2, edu2, A, None, A.shape[0])
        edF = rounded((edF[0].reshape(B, nl, k), edF[1].reshape(B, nl, k)), dF, us)
        edXl, edW = _fm_backward_bounds(dF, edF, Xl, sf["eX"], W, P, sf["eP"], rnd, us)
        gl = dict(dW=edW, dA=edA, dgamma=edg)
        dFm, _ = fm_backward(dF, Xl, W, P, rnd)
        if lay.get("L") is not None:              # linear compression block
            Lm = np.asarray(lay["L"], np.float64)
            Xt = _T(Xl)
            dL_, edL_ = duR[:, nF:], (eduR[0][:, nF:], eduR[1][:, nF:])
            sb, mb = _add(matmul_err(dL_, edL_, Xt, None, 0), matmul_err(dL_, None, Xt, _Te(sf["eX"]), 0))
            gl["dL"] = (np.sqrt(_sq(sb).sum(0) + B * d * UA * UA * _sq((np.abs(dL_) @ np.abs(Xt)).sum(0))),
                        mb.max(0))
            LTb = np.broadcast_to(Lm.T[None], (B,) + Lm.T.shape)
            edXl = _add(edXl, matmul_err(LTb, None, dL_, edL_, Lm.shape[0]))
            dFm = dFm + LTb @ dL_
        if lay.get("C") is not None:
            C = np.asarray(lay["C"], np.float64)
            Xt = _T(Xl)
            # dC = sum_b duR_b X_b^T
            sb, mb = _add(matmul_err(duR, eduR, Xt, None, 0), matmul_err(duR, None, Xt, _Te(sf["eX"]), 0))
            gl["dC"] = (np.sqrt(_sq(sb).sum(0) + B * d * UA * UA * _sq((np.abs(duR) @ np.abs(Xt)).sum(0))),
                        mb.max(0))
            CTb = np.broadcast_to(C.T[None], (B,) + C.T.shape)
            edXl = _add(edXl, matmul_err(CTb, None, duR, eduR, nv))
            dY = dFm + CTb @ duR
        else:
            edXl = _add(edXl, edu)
            dY = dFm + du
        grads[li] = gl
        edY = edXl
    return edY, grads


def stack_bounds(X, eX, dY, edY, layers, caches, dtype):
    """(s, m) of the stacked interaction evaluated on its own: output, input
    gradient and per-layer parameter gradients, for inputs X and dY with
    scales eX and edY (zeros: identical inputs on both sides)."""
    from .step import rounding
    rnd, us = rounding(dtype), storage_unit(dtype)
    d = X.shape[2]
    e_out, st_fwd = _stack_forward_bounds(layers, caches, eX, d, rnd, us)
    edX, grads = _stack_backward_bounds(layers, caches, st_fwd, dY, edY, rnd, us)
    return e_out, edX, grads


def step_bounds(cfg, params, table, batch, c, g, lr_tables=None, loss_normalizer=None):
    """(s, m) of accelerator - oracle for the outputs of ``step.step``
    (``c``: forward cache, ``g``: gradients), keyed like them: X, t (top
    input), logits, loss, dz, d_top_in, top_dW/top_db (lists),
    bottom_dW/bottom_db, fm_dW, stack (list of dicts), dX_emb, grad_rows,
    updated_rows."""
    from .step import rounding
    rnd = rounding(cfg.dtype)
    us = storage_unit(cfg.dtype)
    B, F, d = int(cfg.B), int(cfg.F), int(cfg.d)
    n, s0 = cfg.n_slots, cfg.first_emb_slot
    out = {}
    X = c["X"]
    tab = np.asarray(table, np.float64)
    mean = lambda x: x.mean(-1, keepdims=True)
    mx = lambda x: x.max(-1, keepdims=True)

    # ---- forward ---------------------------------------------------------
    lengths = np.diff(np.asarray(batch["offsets"], np.int64)).reshape(F, B).T.astype(np.float64)
    absP = pool_forward(np.abs(tab), batch["row_base"], batch["offsets"], batch["indices"], F, B, cfg.pool)
    sX, mX = np.zeros_like(X), np.zeros_like(X)
    sX[:, s0:], mX[:, s0:] = rounded((np.sqrt(lengths[..., None] + 3) * UA * absP, 0.0), X[:, s0:], us)
    if cfg.has_dense:
        hsb = c["hs_bottom"]
        ehb, preb = _mlp_forward_bounds(hsb, params["bottom"], None, us, last_linear=False)
        sX[:, 0], mX[:, 0] = ehb[-1]
    eX = (sX, mX)
    out["X"] = eX
    head = [(sX[:, 0], mX[:, 0])] if cfg.has_dense else []
    if cfg.interact == "dot":
        i, j = pair_indices(n)
        sG, mG = matmul_err(X, eX, _T(X), _Te(eX), d)
        e_inter = rounded((sG[:, i, j], mG[:, i, j]), c["inter"], us)
    elif cfg.interact == "fm":
        W = np.asarray(params["fm_W"], np.float64)
        O = c["inter"].reshape(B, n, -1)
        eP, eO = _fm_forward_bounds(X, eX, W, c["fm_P"], O, us)
        e_inter = (eO[0].reshape(B, -1), eO[1].reshape(B, -1))
    else:
        eXl, st_fwd = _stack_forward_bounds(params["stack"], c["stack"], eX, d, rnd, us)
        e_inter = (eXl[0].reshape(B, -1), eXl[1].reshape(B, -1))
    et = (np.concatenate([h[0] for h in head] + [e_inter[0]], axis=1),
          np.concatenate([h[1] for h in head] + [e_inter[1]], axis=1))
    out["t"] = et
    hst = c["hs_top"]
    eht, pret = _mlp_forward_bounds(hst, params["top"], et, us, last_linear=True)
    ez = eht[-1]
    out["logits"] = ez

    # ---- loss --------------------------------------------------------------
    z = c["logits"]
    y = np.asarray(batch["labels"], np.float64)
    m = np.asarray(batch["mask"], np.float64)
    N = max(1.0, float(m.sum())) if loss_normalizer is None else float(loss_normalizer)
    sig = sigmoid(z)
    edz = (m * np.sqrt(_sq(ez[0] / 4.0) + _sq(8 * UA)) / N, m * ez[1] / 4.0 / N)   # sigmoid' <= 1/4
    out["dz"] = edz
    l = np.maximum(z, 0) - z * y + np.log1p(np.exp(-np.abs(z)))
    out["loss"] = (np.array([np.sqrt(np.sum(_sq(m * np.abs(sig - y) * ez[0]))
                                     + np.sum(_sq(m * 8 * UA * (np.abs(z) + np.abs(z * y) + 1)))
                                     + m.size * UA * UA * _sq(np.sum(m * l))) / N]),
                   np.array([float(np.max(m * ez[1], initial=0.0)) / N]))

    # ---- backward ----------------------------------------------------------
    gz = rnd(c["dz"])
    egz = rounded(edz, gz, us)
    dWt, dbt, dt_raw, edt_raw = _mlp_backward_bounds(gz, egz, hst, eht, c["masks_top"], pret,
                                                     params["top"], rnd, us, need_input=True)
    out["top_dW"], out["top_db"] = dWt, dbt
    gt = rnd(dt_raw)
    egt = rounded(edt_raw, gt, us)
    out["d_top_in"] = egt
    off = d if cfg.has_dense else 0
    if cfg.interact == "dot":
        i, j = pair_indices(n)
        S = np.zeros((B, n, n))
        S[:, i, j] = gt[:, off:]
        S[:, j, i] = gt[:, off:]
        eS = (np.zeros((B, n, n)), np.zeros((B, n, n)))
        for q in range(2):
            eS[q][:, i, j] = egt[q][:, off:]
            eS[q][:, j, i] = egt[q][:, off:]
        edXi = matmul_err(S, eS, X, eX, n)
    elif cfg.interact == "fm":
        W = np.asarray(params["fm_W"], np.float64)
        k = W.shape[1]
        G = gt[:, off:].reshape(B, n, k)
        eG = (egt[0][:, off:].reshape(B, n, k), egt[1][:, off:].reshape(B, n, k))
        edXi, out["fm_dW"] = _fm_backward_bounds(G, eG, X, eX, W, c["fm_P"], eP, rnd, us)
    else:
        edY = (egt[0].reshape(B, cfg.stack_n, d), egt[1].reshape(B, cfg.stack_n, d))
        edY, out["stack"] = _stack_backward_bounds(params["stack"], c["stack"], st_fwd,
                                                   gt.reshape(B, cfg.stack_n, d), edY, rnd, us)
        edXi = edY
    out["dX_emb"] = rounded((edXi[0][:, s0:], edXi[1][:, s0:]), g["dX_emb"], us)
    if cfg.has_dense:
        if cfg.interact == "dot":
            dXi0 = dot_backward(gt[:, d:], X)[:, 0]
        else:
            dXi0 = fm_backward(gt[:, d:].reshape(B, n, cfg.fm_rank), X, params["fm_W"], c["fm_P"], rnd)[0][:, 0]
        dh = dXi0 + gt[:, :d]
        edh = _add((edXi[0][:, 0], edXi[1][:, 0]), (egt[0][:, :d], egt[1][:, :d]), (UA * np.abs(dh), 0.0))
        a, ea = preb[-1]
        mask = c["masks_bottom"][-1]
        gb = rnd(dh * mask)
        egb = rounded(_masked(dh, edh, mask, a, ea), gb, us)
        dWb, dbb, _, _ = _mlp_backward_bounds(gb, egb, hsb, ehb, c["masks_bottom"], preb,
                                              params["bottom"], rnd, us, need_input=False)
        out["bottom_dW"], out["bottom_db"] = dWb, dbb

    # ---- sparse gradient and SGD ---------------------------------------------
    dXe = g["dX_emb"]
    rb, off_, idx = batch["row_base"], batch["offsets"], batch["indices"]
    sE, mE = out["dX_emb"]
    if cfg.pool == "mean":       # each occurrence carries dX / len
        Ln = np.maximum(lengths, 1.0)[..., None]
        sE, mE = sE / Ln, mE / Ln
    uniq, vG = pool_backward(_sq(sE), rb, off_, idx, F, B, "sum")
    _, aG = pool_backward(np.abs(dXe), rb, off_, idx, F, B, cfg.pool)
    # the largest single jump among a row's occurrences
    keys = row_keys(rb, off_, idx, F, B)
    pos = np.searchsorted(uniq, keys)
    bag = np.repeat(np.arange(F * B), np.diff(np.asarray(off_, np.int64)))
    mG = np.zeros((uniq.size, d))
    np.maximum.at(mG, pos, mE[bag % B, bag // B])
    counts = g["bookkeeping"]["counts"].astype(np.float64)[:, None]
    eGr = (np.sqrt(vG + (counts + 3) * UA * UA * _sq(aG)), mG)
    out["grad_rows"] = eGr
    lr = cfg.lr_tables if lr_tables is None else lr_tables
    if lr:
        E0 = tab[g["unique_rows"]]
        v = E0 - lr * g["grad_rows"]
        out["updated_rows"] = rounded(_add(_scale(eGr, lr), (2 * UA * np.abs(v), 0.0)), g["updated_rows"], us)
    return out
