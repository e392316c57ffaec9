"""Linear layers with bias and ReLU (or SwishRN): the dense feature processor
("bottom" MLP, Section 3.3.1) and the task modules ("top" MLP with one output
per objective, Section 3.3.3).

Test infrastructure only (see the package docstring).

Weights are ``[out, in]``.  Forward of one layer: ``a = h W^T + b``; a hidden
layer stores ``rnd(max(a, 0))`` (its ReLU output at the storage precision); the
last top layer returns the logits ``a`` unrounded.  Backward of one layer,
given the gradient ``g`` of its output: ``dW = g^T h``, ``db = sum_b g``,
``dh = g W``; the gradient reaching a hidden activation is masked by that
activation being positive (ReLU) and stored as ``rnd(...)``.

SwishRN layers (Section 3.3.4, ``swishrn``) replace the ReLU: the layer
stores its pre-activation ``rnd(a)`` and its output ``rnd(swishrn(a))``; in
the backward the gradient of the output is stored as ``rnd(g W)`` and the
gradient of the pre-activation as ``rnd(swishrn.backward(...))``, and the
gains get their gradients from the stored output gradient.
"""
import numpy as np

from . import fp8 as _fp8
from . import swishrn as _swishrn


def linear(h, W, b):
    return np.asarray(h, np.float64) @ np.asarray(W, np.float64).T + np.asarray(b, np.float64)


def linear_grads(g, h, W):
    """(dW, db, dh) of ``a = h W^T + b`` given ``g = dL/da``."""
    g = np.asarray(g, np.float64)
    h = np.asarray(h, np.float64)
    return g.T @ h, g.sum(axis=0), g @ np.asarray(W, np.float64)


def untied_linear(h, W, b, domain):
    """Parameter untying (Section 3.3.4): W ``[D, out, in]``, b ``[D, out]``;
    sample r uses set ``domain[r]``."""
    h = np.asarray(h, np.float64)
    a = np.empty((h.shape[0], np.shape(W)[1]))
    for g in range(np.shape(W)[0]):
        r = np.asarray(domain) == g
        a[r] = linear(h[r], W[g], b[g])
    return a


def untied_linear_grads(g, h, W, domain):
    """(dW [D, out, in], db [D, out], dh) of ``untied_linear``: each set's
    gradients sum over its own samples only."""
    g, h, W = (np.asarray(x, np.float64) for x in (g, h, W))
    dW, db = np.zeros(W.shape), np.zeros(W.shape[:2])
    dh = np.zeros(h.shape)
    for k in range(W.shape[0]):
        r = np.asarray(domain) == k
        dW[k], db[k], dh[r] = linear_grads(g[r], h[r], W[k])
    return dW, db, dh


def grouped_linear(h, W, b):
    """Per-objective towers' heads (Section 3.3.3): W is ``[T, H]`` and output
    t reads only its tower's inputs ``h[:, t*H:(t+1)*H]``:
    ``a[:, t] = h[:, t*H:(t+1)*H] W[t] + b[t]``."""
    h, W = np.asarray(h, np.float64), np.asarray(W, np.float64)
    T, H = W.shape
    assert h.shape[1] == T * H
    return np.einsum("bth,th->bt", h.reshape(-1, T, H), W) + np.asarray(b, np.float64)


def grouped_linear_grads(g, h, W):
    """(dW [T, H], db, dh) of ``grouped_linear`` given ``g = dL/da``."""
    g, h, W = (np.asarray(x, np.float64) for x in (g, h, W))
    T, H = W.shape
    h3 = h.reshape(-1, T, H)
    return np.einsum("bt,bth->th", g, h3), g.sum(axis=0), (g[:, :, None] * W[None]).reshape(-1, T * H)


def relu_band(h, W, b):
    """Half-width of the band around zero inside which the sign of a
    pre-activation is not fixed by fp32 accumulation: the worst-case error of
    summing the ``K`` products plus the bias in any order in fp32,
    ``K * 2^-24 * (sum_k |W_k h_k| + |b|)``."""
    h = np.abs(np.asarray(h, np.float64))
    K = h.shape[1]
    return (K + 1) * 2.0 ** -24 * (h @ np.abs(np.asarray(W, np.float64)).T + np.abs(np.asarray(b, np.float64)))


def linear_fp8(h, W, b):
    """The FP8 forward of a layer (Section 3.5.2): input rows and weight rows
    quantised to e4m3 with row-wise scales, their exact product, plus the
    bias."""
    qa, sa = _fp8.quantize(h, rowwise=True)
    qw, sw = _fp8.quantize(W, rowwise=True)
    return _fp8.linear_fp8(qa, sa, qw, sw, b)


def _swish_fwd(a, act, i, domain):
    """SwishRN of layer i's pre-activation, per domain when its gains are
    untied ([D, out])."""
    ga, gb = act["gains"][i]
    if np.ndim(ga) == 1:
        out, _, rho = _swishrn.forward(a, ga, gb, act["block"], act["eps"], act["kind"])
        return out, rho
    out = np.empty_like(a)
    rho = np.empty((a.shape[0], len(_swishrn.groups(a.shape[1], act["block"]))))
    for k in range(ga.shape[0]):
        r = np.asarray(domain) == k
        out[r], _, rho[r] = _swishrn.forward(a[r], ga[k], gb[k], act["block"], act["eps"], act["kind"])
    return out, rho


def mlp_forward(h0, layers, rnd, relu_last, overrides=None, fp8_layers=(), act=None, grouped_last=False,
                domain=None):
    """Returns ``(hs, masks)``: the layer inputs/outputs ``[h0, h1, ..., hL]``
    and, per layer, its ReLU decision (``None`` for a linear last layer).
    Every layer but (optionally) the last applies ReLU and storage rounding.

    ``overrides[i]``, when given, is ``(where, positive)``: at the positions in
    ``where`` the ReLU of layer i takes the decision ``positive`` instead of
    the sign of the float64 pre-activation.  Parity tests use it only inside
    ``relu_band``, where either decision is a correct result of fp32
    arithmetic.  Layers listed in ``fp8_layers`` run their forward product
    in FP8 (``linear_fp8``).

    ``act`` (optional) makes the activated layers SwishRN layers: a dict with
    ``kind`` ("sigmoid" | "hard"), ``block`` (0: RMSNorm over the row; b:
    BlockNorm groups of b features), ``eps`` and ``gains`` (per layer
    ``(ga, gb)``).  Their entry in the returned list is then a dict
    ``{"pre": a, "rho": ...}`` instead of a ReLU mask.  ``grouped_last``:
    the last (linear) layer is the towers' heads (``grouped_linear``).
    Layers whose W is ``[D, out, in]`` are untied (``untied_linear``, and
    their SwishRN gains ``[D, out]``) over the per-sample ``domain``."""
    hs = [np.asarray(h0, np.float64)]
    masks = []
    for i, (W, b) in enumerate(layers):
        last = i == len(layers) - 1
        if grouped_last and last:
            a = grouped_linear(hs[-1], W, b)
        elif np.ndim(W) == 3:
            a = untied_linear(hs[-1], W, b, domain)
        else:
            a = linear_fp8(hs[-1], W, b) if i in fp8_layers else linear(hs[-1], W, b)
        if act is not None and (relu_last or not last):
            out, rho = _swish_fwd(a, act, i, domain)
            hs.append(rnd(out))
            masks.append({"pre": a, "rho": rho})
        elif relu_last or not last:
            on = a > 0
            if overrides is not None and overrides[i] is not None:
                where, positive = overrides[i]
                on = np.where(where, positive, on)
            hs.append(rnd(np.where(on, np.maximum(a, 0.0), 0.0)))
            masks.append(on)
        else:
            hs.append(a)
            masks.append(None)
    return hs, masks


def mlp_backward(g_out, hs, masks, layers, rnd, relu_last, need_input_grad, act=None, dgains=None,
                 grouped_last=False, domain=None):
    """Backward through ``mlp_forward``.  ``g_out`` is dL/d(hs[-1]) (before the
    last ReLU mask when ``relu_last``).  Returns (dWs, dbs, dL/dh0 or None).
    With ``act`` (as in ``mlp_forward``) the gain gradients of the SwishRN
    layers go to ``dgains[i] = (dga, dgb)``; ``act["overrides"][i]``, when
    given, is layer i's ``swishrn.backward`` gate-derivative override."""
    L = len(layers)

    def through(i, g):
        """Gradient of layer i's pre-activation from that of its output."""
        if act is None:
            return rnd(g * masks[i])
        ga, gb = act["gains"][i]
        go = rnd(g)
        ov = (act.get("overrides") or {}).get(i)
        if np.ndim(ga) == 1:
            dh, dga, dgb = _swishrn.backward(go, masks[i]["pre"], ga, gb, act["block"], act["eps"], act["kind"],
                                             grad_override=ov)
        else:                                   # untied gains: each domain's rows
            dh, dga, dgb = np.empty_like(go), np.zeros(ga.shape), np.zeros(gb.shape)
            for k in range(ga.shape[0]):
                r = np.asarray(domain) == k
                ovk = None if ov is None else (ov[0][r], ov[1][r])
                dh[r], dga[k], dgb[k] = _swishrn.backward(go[r], masks[i]["pre"][r], ga[k], gb[k], act["block"],
                                                          act["eps"], act["kind"], grad_override=ovk)
        if dgains is not None:
            dgains[i] = (dga, dgb)
        return rnd(dh)

    g = np.asarray(g_out, np.float64)
    if relu_last:
        g = through(L - 1, g)
    dWs, dbs = [None] * L, [None] * L
    dh0 = None
    for i in range(L - 1, -1, -1):
        W, _ = layers[i]
        if grouped_last and i == L - 1:
            dW, db, dh = grouped_linear_grads(g, hs[i], W)
        elif np.ndim(W) == 3:
            dW, db, dh = untied_linear_grads(g, hs[i], W, domain)
        else:
            dW, db, dh = linear_grads(g, hs[i], W)
        dWs[i], dbs[i] = dW, db
        if i > 0:
            g = through(i - 1, dh)
        elif need_input_grad:
            dh0 = dh
    return dWs, dbs, dh0
