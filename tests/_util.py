"""Shared helpers of the GPU parity tests (test infrastructure)."""
import numpy as np
import torch

import synth
from oracle import bounds as obounds
from oracle import embbag as oembbag
from oracle import fp8 as ofp8
from oracle import interact as ointeract
from oracle import loss as oloss
from oracle import mlp as omlp
from oracle import step as ostep
from oracle import swishrn as oswish
from oracle.metrics import max_rel_err, max_rel_err_normwise

DEV = "cuda"


def tol(cfg):
    """fp32 workloads: 1e-5; bf16-storage workloads: 2e-2 (max relative error)."""
    return 1e-5 if cfg.dtype == "f32" else 2e-2


def assert_close(name, got, ref, t):
    got = got.detach().float().cpu().numpy() if torch.is_tensor(got) else np.asarray(got)
    err = max_rel_err(got, ref)
    print(f"  {name}: max_rel_err={err:.3e} (tol {t:.0e})", flush=True)
    assert err <= t, f"{name}: max_rel_err {err} > {t}"


def _np64(x):
    if torch.is_tensor(x):
        return x.detach().float().cpu().double().numpy()
    return np.asarray(x, np.float64)


def _row_floor(ref):
    """max(|r|, rms of r's last-axis row), the element-wise metric's scale."""
    rr = ref.reshape(1, -1) if ref.ndim <= 1 else ref.reshape(-1, ref.shape[-1])
    rms = np.sqrt(np.mean(rr * rr, axis=-1, keepdims=True))
    return np.maximum(np.abs(rr), rms).reshape(ref.shape)


def assert_close_derived(name, got, ref, e, t):
    """A tensor of the composed step (downstream of several bf16 storage
    points), compared element by element: an element passes when it is
    within t of its reference by the element-wise metric (scale max(|r|,
    row rms)), or within the accepted deviation ``oracle.bounds.allowed(e)``
    that the arithmetic itself allows that element (the spread between two
    correct evaluations that round differently); the normwise error must
    also meet t.  fp32 workloads: the strict metric at t."""
    got, ref = _np64(got), np.asarray(ref, np.float64)
    assert got.shape == ref.shape, (name, got.shape, ref.shape)
    if t <= 1e-5:
        err = max_rel_err(got, ref)
        print(f"  {name}: max_rel_err={err:.3e} (tol {t:.0e})", flush=True)
        assert err <= t, f"{name}: max_rel_err {err} > {t}"
        return
    assert np.all(np.isfinite(got)), f"{name}: non-finite values"
    norm = max_rel_err_normwise(got, ref)
    diff = np.abs(got - ref)
    strict_ok = diff <= t * _row_floor(ref)
    acc = obounds.allowed(e)
    derived_ok = diff <= acc
    bad = ~(strict_ok | derived_ok)
    n_der = int(np.count_nonzero(~strict_ok & derived_ok))
    worst = float(np.max(diff / np.maximum(acc, 1e-300), initial=0.0))
    print(f"  {name}: normwise={norm:.3e} (tol {t:.0e}); {n_der} of {diff.size} elements beyond "
          f"{t:.0e} and within the derived deviation (worst |x-r|/allowed {worst:.2f})", flush=True)
    assert norm <= t, f"{name}: normwise max relative error {norm} > {t}"
    if bad.any():
        i = np.unravel_index(np.argmax(np.where(bad, diff / np.maximum(acc, 1e-300), 0)), diff.shape)
        raise AssertionError(f"{name}: {int(bad.sum())} elements outside both the element-wise "
                             f"tolerance and the derived deviation; worst at {i}: got {got[i]}, "
                             f"ref {ref[i]}, allowed {acc[i]}")


def assert_product(name, got, ref, absref, K, storage_unit=None, t=2e-2):
    """One stage recomputed by the oracle from the accelerator's own stored
    operands: ``ref`` is the exact result, ``absref`` the same product of
    absolute values and ``K`` the number of terms per element.  An fp32 sum
    of K terms in any order is within (K+3) 2^-24 absref of the exact value
    (bf16 x bf16 products are exact in fp32); a result stored at storage
    unit ``us`` adds one rounding, us (|ref| + that).  Every element must
    meet this bound, and the tensor the element-wise metric at t."""
    got, ref, absref = _np64(got), np.asarray(ref, np.float64), np.asarray(absref, np.float64)
    assert got.shape == ref.shape, (name, got.shape, ref.shape)
    acc = (K + 3) * 2.0 ** -24 * absref
    bound = acc + (storage_unit * (np.abs(ref) + acc) if storage_unit else 0.0) + 1e-37
    ratio = float(np.max(np.abs(got - ref) / bound, initial=0.0))
    err = max_rel_err(got, ref)
    print(f"  {name} [stage]: max_rel_err={err:.3e} (tol {t:.0e}), worst |x-r|/bound={ratio:.3f}", flush=True)
    assert np.all(np.isfinite(got)), f"{name}: non-finite values"
    assert ratio <= 1.0, f"{name}: outside the fp32 accumulation bound (ratio {ratio})"
    assert err <= t, f"{name}: max_rel_err {err} > {t}"


def assert_fp8_layer(name, got, h, W, b, fast, t=2e-2):
    """A hidden layer whose forward product ran in FP8 (row-wise e4m3 input
    and weights): within oracle.fp8.linear_fp8_bound of the exact product of
    the codes the oracle takes from the same stored input, plus bf16 output
    rounding (ReLU is 1-Lipschitz)."""
    qa, sa = ofp8.quantize(h, rowwise=True)
    qw, sw = ofp8.quantize(W, rowwise=True)
    ref = ofp8.linear_fp8(qa, sa, qw, sw, b, relu=True)
    bound = ofp8.linear_fp8_bound(qa, sa, qw, sw, b, fast_accum=fast)
    bound = bound + 2.0 ** -8 * (np.abs(ref) + bound) + 1e-37
    got = _np64(got)
    ratio = float(np.max(np.abs(got - ref) / bound, initial=0.0))
    err = max_rel_err(got, ref)
    print(f"  {name} [fp8 stage]: max_rel_err={err:.3e}, worst |x-r|/bound={ratio:.3f}", flush=True)
    assert np.all(np.isfinite(got)) and ratio <= 1.0, f"{name}: outside the fp8 bound ({ratio})"
    if not fast:
        assert err <= t, f"{name}: max_rel_err {err} > {t}"


def assert_bounded(name, got, ref, e, storage_unit=None, t=2e-2):
    """Element-wise: |got - ref| <= e (+ one rounding to the storage grid,
    us (|ref| + e)), and the element-wise metric at t."""
    got, ref, e = _np64(got), np.asarray(ref, np.float64), np.asarray(e, np.float64)
    assert got.shape == ref.shape, (name, got.shape, ref.shape)
    bound = e + (storage_unit * (np.abs(ref) + e) if storage_unit else 0.0) + 1e-37
    ratio = float(np.max(np.abs(got - ref) / bound, initial=0.0))
    err = max_rel_err(got, ref)
    print(f"  {name} [stage]: max_rel_err={err:.3e} (tol {t:.0e}), worst |x-r|/bound={ratio:.3f}", flush=True)
    assert np.all(np.isfinite(got)), f"{name}: non-finite values"
    assert ratio <= 1.0, f"{name}: outside the derived bound (ratio {ratio})"
    assert err <= t, f"{name}: max_rel_err {err} > {t}"


def check_swishrn_forward(name, cfg, act, i, h, W, b, pre, rinv, out, us, t):
    """A SwishRN layer's forward from its stored input h: the pre-activation
    (a product), then the activation -- from the exact pre-activation within
    the GEMM's accumulation error when bf16 models normalise in the GEMM's
    epilogue (BlockNorm), else from the stored pre-activation -- and rho."""
    ga, gb = act["gains"][i]
    a = h @ W.T + b
    ab = np.abs(h) @ np.abs(W).T + np.abs(b)
    K = W.shape[1] + 1
    assert_product(f"{name} pre-activation", pre, a, ab, K, us, t)
    if cfg.dtype == "bf16" and act["block"] == 128:
        src, eh = a, (K + 3) * 2.0 ** -24 * ab
    else:
        src, eh = _np64(pre), 0.0
    ref, _, rho = oswish.forward(src, ga, gb, act["block"], act["eps"], act["kind"])
    e_out, e_rho = oswish.forward_bound(src, eh, ga, gb, act["block"], act["eps"], act["kind"])
    assert_bounded(f"{name} SwishRN", out, ref, e_out, us, t)
    assert_bounded(f"{name} rho", rinv, rho, e_rho, None, t)


def check_swishrn_backward(name, act, i, gout, pre, rinv, dh, us, t):
    """A SwishRN layer's backward chain from its stored output gradient,
    pre-activation and rho."""
    ga, gb = act["gains"][i]
    gout, pre, rinv = _np64(gout), _np64(pre), _np64(rinv)
    ref, _, _ = oswish.backward(gout, pre, ga, gb, act["block"], act["eps"], act["kind"], rho=rinv)
    e, _, _ = oswish.backward_bound(gout, 0.0, pre, ga, gb, act["block"], act["eps"], act["kind"], rinv)
    assert_bounded(f"{name} SwishRN backward", dh, ref, e, us, t)


def check_swishrn_gains(name, act, i, gout, pre, rinv, dgain, t):
    ga, gb = act["gains"][i]
    gout, pre, rinv = _np64(gout), _np64(pre), _np64(rinv)
    _, dga, dgb = oswish.backward(gout, pre, ga, gb, act["block"], act["eps"], act["kind"], rho=rinv)
    _, e_a, e_b = oswish.backward_bound(gout, 0.0, pre, ga, gb, act["block"], act["eps"], act["kind"], rinv)
    dg = _np64(dgain)
    assert_bounded(f"{name}.dga", dg[0], dga, e_a, None, t)
    assert_bounded(f"{name}.dgb", dg[1], dgb, e_b, None, t)


def check_stages(cfg, params, batch, v, grads, rows=None, wgrad_rows=None, fp8_top=None):
    """Stage-wise parity of one step: every stage recomputed in float64 by
    the oracle from the accelerator's own stored inputs of that stage, so the
    only admissible difference is that stage's own arithmetic.  v: the step's
    workspace views; grads: the accelerator's parameter gradients (dict:
    top_dW/top_db/bottom_dW/bottom_db lists, fm_dW, stack list of dicts);
    rows (optional): samples for the per-sample stages (all if None);
    wgrad_rows (optional): dict ("top"|"bottom", layer) -> output rows of
    that weight gradient to recompute over the whole batch (all if absent).
    Sample-summed interaction gradients are checked when rows is None.
    fp8_top ("precise" / "fast"): the top MLP's hidden layers ran their
    forward product in FP8 (assert_fp8_layer)."""
    us = 2.0 ** -8 if cfg.dtype == "bf16" else None
    t = tol(cfg)
    B, d = cfg.B, cfg.d
    R = np.arange(B) if rows is None else np.asarray(rows)
    wr = wgrad_rows or {}
    L = len(params["top"])
    tin = _np64(v["t"][:, :cfg.top_in])
    h_top = [tin] + [_np64(a) for a in v["top_act"]]
    g_top = [_np64(g) for g in v["top_grad"]]
    act = ostep.top_act(cfg, params)
    # top MLP forward, layer by layer from the stored inputs
    towers = bool(getattr(cfg, "towers", 0))
    # the heads' products: dense, or the towers' grouped heads (objective t
    # reads only its tower's units)
    def heads_fwd(h, W, b):
        return omlp.grouped_linear(h, W, b) if towers else h @ W.T + b

    def heads_dgrad(g, W):
        return omlp.grouped_linear_grads(g, np.zeros((g.shape[0], W.size)), W)[2] if towers else g @ W

    def heads_wgrad(g, h, W):
        return omlp.grouped_linear_grads(g, h, W)[0] if towers else g.T @ h

    dom = np.asarray(batch.get("domain", np.zeros(B, np.int64)))

    def parts(i, rows_sel):
        """(params of layer i, act view, row subset) per domain for an untied
        layer (W [D, out, in]), else one part with the whole row set."""
        W, b = (np.asarray(x, np.float64) for x in params["top"][i])
        if W.ndim == 2:
            return [(W, b, act, rows_sel)]
        out = []
        for k in range(W.shape[0]):
            sel = rows_sel[dom[rows_sel] == k]
            av = None
            if act is not None:
                av = dict(act, gains=list(act["gains"]))
                ga, gb = act["gains"][i]
                av["gains"][i] = (ga[k], gb[k])
            if sel.size:
                out.append((W[k], b[k], av, sel))
        return out

    def untied_at(i):
        return np.ndim(params["top"][i][0]) == 3

    for i in range(L):
        last = i == L - 1
        for W, b, av, Rp in parts(i, R):
            h = h_top[i][Rp]
            a = heads_fwd(h, W, b) if last else h @ W.T + b
            ab = heads_fwd(np.abs(h), np.abs(W), np.abs(b)) if last else np.abs(h) @ np.abs(W).T + np.abs(b)
            if i < L - 1 and av is not None:
                check_swishrn_forward(f"top{i}", cfg, av, i, h, W, b, _np64(v["top_pre"][i])[Rp],
                                      _np64(v["top_rinv"][i])[Rp], h_top[i + 1][Rp], us, t)
            elif i < L - 1 and fp8_top:
                assert_fp8_layer(f"top{i} forward", h_top[i + 1][Rp], h, W, b, fp8_top == "fast", t)
            elif i < L - 1:
                assert_product(f"top{i} forward", h_top[i + 1][Rp], np.maximum(a, 0), ab, W.shape[1] + 1, us, t)
            else:
                assert_product("logits", _np64(v["logits"])[Rp], a, ab, W.shape[1] + 1, None, t)
    # loss and dz from the stored logits
    z = _np64(v["logits"])
    N = max(1.0, float(np.asarray(batch["mask"]).sum()))
    L_ref, dz_ref = oloss.masked_bce(z, batch["labels"], batch["mask"], N)
    e_loss = max_rel_err(_np64(v["loss"]), np.array([L_ref]))
    e_dz = max_rel_err(_np64(v["d_logits"]), dz_ref)
    print(f"  loss [stage]: {e_loss:.3e}; d_logits [stage]: {e_dz:.3e} (tol 1e-5)", flush=True)
    assert e_loss <= 1e-5 and e_dz <= 1e-5
    # the gradient chain: g_{i-1} = (g_i W_i) masked by the stored h_i > 0
    # (SwishRN: g_i W_i is the stored output gradient, taken through the
    # SwishRN backward); untied layers per domain
    for i in range(L - 1, -1, -1):
        # parameter views of layer i and, for the activation below, layer i-1
        lower = parts(i - 1, R) if i > 0 and untied_at(i - 1) else None
        for W, _, _, Rp in parts(i, R):
            subs = [(Rp, act)] if lower is None else [(np.intersect1d(Rp, q[3]), q[2]) for q in lower]
            for Rq, av in subs:
                if Rq.size == 0:
                    continue
                if i == L - 1:
                    prod, ab = heads_dgrad(g_top[i][Rq], W), heads_dgrad(np.abs(g_top[i][Rq]), np.abs(W))
                    Kc = 1 if towers else W.shape[0]
                else:
                    prod, ab, Kc = g_top[i][Rq] @ W, np.abs(g_top[i][Rq]) @ np.abs(W), W.shape[0]
                if i > 0 and av is not None:
                    gout = _np64(v["top_gout"][i - 1])[Rq]
                    assert_product(f"top{i} output grad", gout, prod, ab, Kc, us, t)
                    check_swishrn_backward(f"top{i - 1}", av, i - 1, gout, _np64(v["top_pre"][i - 1])[Rq],
                                           _np64(v["top_rinv"][i - 1])[Rq], g_top[i - 1][Rq], us, t)
                elif i > 0:
                    on = h_top[i][Rq] > 0
                    assert_product(f"top{i} grad chain", g_top[i - 1][Rq], prod * on, ab * on, Kc, us, t)
                else:
                    assert_product("d_t", tin_grad(v, cfg)[Rq], prod, ab, Kc, us, t)
    # weight and bias gradients from the stored chain and activations (an
    # untied layer: each domain's set from its own samples)
    allrows = np.arange(B)
    for i in range(L):
        r = wr.get(("top", i), slice(None))
        if i == L - 1 and towers:
            Wl = np.asarray(params["top"][i][0], np.float64)
            gi, hi = g_top[i], h_top[i]
            assert_product(f"top{i}.dW (towers)", _np64(grads["top_dW"][i]), heads_wgrad(gi, hi, Wl),
                           heads_wgrad(np.abs(gi), np.abs(hi), Wl), B, None, t)
            assert_product(f"top{i}.db", _np64(grads["top_db"][i]), gi.sum(0), np.abs(gi).sum(0), B, None, t)
            continue
        dWg, dbg = _np64(grads["top_dW"][i]), _np64(grads["top_db"][i])
        for k, (_, _, _, Rp) in enumerate(parts(i, allrows)):
            gi, hi = g_top[i][Rp][:, r], h_top[i][Rp]
            dW_k = dWg[k] if untied_at(i) else dWg
            db_k = dbg[k] if untied_at(i) else dbg
            tag = f"top{i}[domain {k}]" if untied_at(i) else f"top{i}"
            assert_product(f"{tag}.dW", dW_k[r], gi.T @ hi, np.abs(gi).T @ np.abs(hi), Rp.size, None, t)
            assert_product(f"{tag}.db", db_k[r], gi.sum(0), np.abs(gi).sum(0), Rp.size, None, t)
    if act is not None and rows is None:
        for i in range(L - 1):
            dgk = _np64(grads["top_dgain"][i])
            for k, (_, _, av, Rp) in enumerate(parts(i, allrows)):
                check_swishrn_gains(f"top{i}", av, i, _np64(v["top_gout"][i])[Rp], _np64(v["top_pre"][i])[Rp],
                                    _np64(v["top_rinv"][i])[Rp], dgk[k] if untied_at(i) else dgk, t)
    X = _np64(v["X"])
    dX = _np64(v["dX"])
    gt = tin_grad(v, cfg)
    if cfg.has_dense:
        hb = [_np64(batch["dense"])] + [_np64(a) for a in v["bottom_act"]] + [X[:, 0]]
        gb = [_np64(g) for g in v["bottom_grad"]]
        nb = len(params["bottom"])
        for i, (W, b) in enumerate(params["bottom"]):
            W, b = np.asarray(W, np.float64), np.asarray(b, np.float64)
            a = hb[i][R] @ W.T + b
            assert_product(f"bottom{i} forward", hb[i + 1][R], np.maximum(a, 0),
                           np.abs(hb[i][R]) @ np.abs(W).T + np.abs(b), W.shape[1] + 1, us, t)
        # the bottom output's gradient is the stored slot-0 gradient, masked
        assert np.array_equal(gb[nb - 1], dX[:, 0] * (X[:, 0] > 0)), "bottom output gradient"
        for i in range(nb - 1, 0, -1):
            W = np.asarray(params["bottom"][i][0], np.float64)
            on = hb[i][R] > 0
            assert_product(f"bottom{i} grad chain", gb[i - 1][R], (gb[i][R] @ W) * on,
                           (np.abs(gb[i][R]) @ np.abs(W)) * on, W.shape[0], us, t)
        for i in range(nb):
            r = wr.get(("bottom", i), slice(None))
            assert_product(f"bottom{i}.dW", _np64(grads["bottom_dW"][i])[r], gb[i][:, r].T @ hb[i],
                           np.abs(gb[i][:, r]).T @ np.abs(hb[i]), B, None, t)
            assert_product(f"bottom{i}.db", _np64(grads["bottom_db"][i])[r], gb[i][:, r].sum(0),
                           np.abs(gb[i][:, r]).sum(0), B, None, t)
    # the interaction, forward and backward, from the stored X and d_t
    rnd = ostep.rounding(cfg.dtype)
    u_ = us or 2.0 ** -24
    off = d if cfg.has_dense else 0
    Xs, gts, ts, dXs = X[R], gt[R], tin[R], dX[R]
    head = np.zeros_like(Xs)                  # the top input's slot-0 gradient enters dX[:, 0]
    if cfg.has_dense:
        head[:, 0] = gts[:, :d]
    zero = lambda x: (np.zeros(x.shape), np.zeros(x.shape))
    if cfg.interact == "dot":
        n = cfg.n_slots
        i_, j_ = ointeract.pair_indices(n)
        G = Xs @ Xs.transpose(0, 2, 1)
        aG = np.abs(Xs) @ np.abs(Xs).transpose(0, 2, 1)
        assert_product("interaction forward", ts[:, off:], G[:, i_, j_], aG[:, i_, j_], d, us, t)
        S = np.zeros((Xs.shape[0], n, n))
        S[:, i_, j_] = gts[:, off:]
        S[:, j_, i_] = gts[:, off:]
        assert_product("interaction backward dX", dXs, S @ Xs + head,
                       np.abs(S) @ np.abs(Xs) + np.abs(head), n + 1, us, t)
    elif cfg.interact == "fm":
        W = np.asarray(params["fm_W"], np.float64)
        n, k = cfg.n_slots, cfg.fm_rank
        O, P = ointeract.fm_forward(Xs, W, rnd)
        eP, eO = obounds._fm_forward_bounds(Xs, zero(Xs), W, P, O, u_)
        nr = O.shape[0]
        assert_close_derived("interaction forward [stage]", ts[:, off:], O.reshape(nr, -1),
                             (eO[0].reshape(nr, -1), eO[1].reshape(nr, -1)), t)
        G = gts[:, off:].reshape(-1, n, k)
        dXr, dWr = ointeract.fm_backward(G, Xs, W, P, rnd)
        edX, edW = obounds._fm_backward_bounds(G, zero(G), Xs, zero(Xs), W, P, eP, rnd, u_)
        full = dXr + head
        assert_close_derived("interaction backward dX [stage]", dXs, rnd(full), obounds.rounded(edX, full, u_), t)
        if rows is None:
            assert_close_derived("fm.dW [stage]", grads["fm_dW"], dWr, edW, t)
    elif cfg.stack_fp8 is not None:
        layers = params["stack"]
        dX1, sg, edX, eg = check_stack_fp8(layers, X, v["stack_state"], tin, gt, None, None, cfg.stack_fp8,
                                           cfg.ln_eps, rows=rows, t=t)
        assert_close_derived("stack backward dX [stage]", dXs, rnd(dX1), obounds.rounded(edX, dX1, u_), t)
        if rows is None:
            for l, (gl, el) in enumerate(zip(sg, eg)):
                for key in gl:
                    assert_close_derived(f"stack{l}.{key} [stage]", grads["stack"][l][key], gl[key], el[key], t)
    else:
        layers = params["stack"]
        XL, caches = ointeract.stack_forward(Xs, layers, cfg.stack_n, d, rnd, cfg.ln_eps)
        dY = gts.reshape(-1, cfg.stack_n, d)
        dX1, sg = ointeract.stack_backward(dY, layers, caches, rnd)
        e_out, edX, eg = obounds.stack_bounds(Xs, zero(Xs), dY, zero(dY), layers, caches, cfg.dtype)
        nr = XL.shape[0]
        assert_close_derived("stack forward [stage]", ts, XL.reshape(nr, -1),
                             (e_out[0].reshape(nr, -1), e_out[1].reshape(nr, -1)), t)
        assert_close_derived("stack backward dX [stage]", dXs, rnd(dX1), obounds.rounded(edX, dX1, u_), t)
        if rows is None:
            for l, (gl, el) in enumerate(zip(sg, eg)):
                for key in gl:
                    assert_close_derived(f"stack{l}.{key} [stage]", grads["stack"][l][key], gl[key], el[key], t)


def check_stack_fp8(layers, X0, state, out, dY, dX, grads, mode, eps, rows=None, t=2e-2):
    """Stage-wise parity of a stacked interaction whose FM projection ran in
    FP8 (Section 3.5.2), from the accelerator's own saved state (per layer
    P, F, H, X_{l+1}; see lattice_interact_state): the projection within
    oracle.fp8.linear_fp8_bound of the exact product of the codes the oracle
    takes from the stored vec(F) and A (the same quantiser, so the same
    codes), the linear compression block within the fp32 sum bound, the
    residual and LayerNorm from the stored H element-wise; then the bf16
    backward through the oracle from those forward values, within the
    derived deviation.  rows: the samples checked (all if None); parameter
    gradients are compared when rows is None."""
    from oracle import fp8 as ofp8
    rnd = ostep.rounding("bf16")
    R = np.arange(X0.shape[0]) if rows is None else np.asarray(rows)
    Xl = _np64(X0)[R]
    X_first = Xl
    L = len(layers)
    d = Xl.shape[2]
    caches = []
    for l, lay in enumerate(layers):
        st = state[l]
        P, F, H = _np64(st["P"])[R], _np64(st["F"])[R], _np64(st["H"])[R]
        Bn = F.shape[0]
        nv = H.shape[1] // d
        vecF = F.reshape(Bn, -1)
        A = np.asarray(lay["A"], np.float64)
        nFd = A.shape[0]
        qf, sf = ofp8.quantize(vecF)
        qa, sa = ofp8.quantize(A)
        ref = ofp8.linear_fp8(qf, sf, qa, sa)
        bound = ofp8.linear_fp8_bound(qf, sf, qa, sa, fast_accum=(mode == "fast")) + 2.0 ** -24 * np.abs(ref)
        ratio = float(np.max(np.abs(H[:, :nFd] - ref) / (bound + 1e-300)))
        print(f"  stack{l} FP8 projection [stage]: worst |x-r|/bound {ratio:.3f}", flush=True)
        assert ratio <= 1.0, f"stack{l}: FP8 projection outside its bound ({ratio})"
        if lay.get("L") is not None:
            Lm = np.asarray(lay["L"], np.float64)
            HL = np.einsum("vu,bud->bvd", Lm, Xl).reshape(Bn, -1)
            aHL = np.einsum("vu,bud->bvd", np.abs(Lm), np.abs(Xl)).reshape(Bn, -1)
            assert_product(f"stack{l} H_L", H[:, nFd:], HL, aHL, Xl.shape[1], None, t)
        C = lay.get("C")
        res = np.einsum("vu,bud->bvd", np.asarray(C, np.float64), Xl) if C is not None else Xl
        u = H.reshape(Bn, nv, d) + res
        mu = u.mean(axis=2, keepdims=True)
        rstd = 1.0 / np.sqrt(((u - mu) ** 2).mean(axis=2, keepdims=True) + eps)
        xhat = (u - mu) * rstd
        y = xhat * np.asarray(lay["gamma"], np.float64)
        got = _np64(out)[R].reshape(Bn, nv, d) if l == L - 1 else _np64(st["Xn"])[R]
        assert_close(f"stack{l} LayerNorm [stage]", got.reshape(Bn, -1), rnd(y).reshape(Bn, -1), t)
        caches.append(dict(X=Xl, P=P, vecF=vecF, xhat=xhat, rstd=rstd))
        Xl = got
    dYr = np.asarray(dY, np.float64)[R].reshape(len(R), -1, d)
    dX1, g = ointeract.stack_backward(dYr, layers, caches, rnd)
    zero = lambda x: (np.zeros(x.shape), np.zeros(x.shape))
    _, edX, eg = obounds.stack_bounds(X_first, zero(X_first), dYr, zero(dYr), layers, caches, "bf16")
    return dX1, g, edX, eg


def tin_grad(v, cfg):
    """The stored gradient of the top input."""
    return _np64(v["d_t"][:, :cfg.top_in])


def grads_of(w):
    """The accelerator's parameter gradients of a Workload, by name."""
    g = dict(top_dW=[L["dW"] for L in w.top], top_db=[L["db"] for L in w.top],
             bottom_dW=[L["dW"] for L in w.bottom], bottom_db=[L["db"] for L in w.bottom],
             fm_dW=w.fm_dW, top_dgain=[L["dgain"] for L in w.top if "dgain" in L])
    if w.stack is not None:
        g["stack"] = [{k: lay[k] for k in ("dW", "dA", "dgamma", "dC", "dL") if lay.get(k) is not None}
                      for lay in w.stack]
    return g


def check_sparse_stage(cfg, batch, v, nnz, E0=None, E1=None, lr=0.0, t=None, sample=None, bk=None):
    """The sparse gradient from the accelerator's own stored dX: integer
    bookkeeping bit-exact, every row gradient within the fp32 sum bound of
    its occurrences, and (with SGD) every updated row within one rounding of
    E0 - lr G on the accelerator's own G; rows that do not occur unchanged.
    sample (optional): indices into the unique rows to recompute (all if
    None); E0 / E1 are then the rows of those samples before / after."""
    t = tol(cfg) if t is None else t
    B, F = cfg.B, cfg.F
    s0 = cfg.first_emb_slot
    if bk is None:
        bk = oembbag.bookkeeping(batch["row_base"], batch["offsets"], batch["indices"], F, B)
    U = int(v["num_unique"].item())
    assert U == bk["unique_rows"].size
    np.testing.assert_array_equal(v["unique_rows"][:U].cpu().numpy(), bk["unique_rows"])
    np.testing.assert_array_equal(v["seg_offsets"][:U + 1].cpu().numpy(), np.append(bk["seg_offsets"], nnz))
    np.testing.assert_array_equal(v["sorted_bags"][:nnz].cpu().numpy(), bk["sorted_bags"])
    if U == 0:
        return
    u_idx = np.arange(U) if sample is None else np.asarray(sample)
    counts, seg = bk["counts"][u_idx], bk["seg_offsets"][u_idx]
    occ = np.concatenate([np.arange(a, a + c) for a, c in zip(seg, counts)])
    bags = bk["sorted_bags"][occ]
    f, b = bags // B, bags % B
    lens = np.diff(np.asarray(batch["offsets"], np.int64))
    dX = v["dX"]
    sel_b = torch.from_numpy(b).to(dX.device)
    sel_s = torch.from_numpy(s0 + f).to(dX.device)
    contrib = _np64(dX[sel_b, sel_s])
    if cfg.pool == "mean":
        contrib = contrib / lens[bags][:, None]
    starts = np.concatenate([[0], np.cumsum(counts)[:-1]])
    G = np.add.reduceat(contrib, starts, axis=0)
    aG = np.add.reduceat(np.abs(contrib), starts, axis=0)
    Gg = _np64(v["grad_rows"][torch.from_numpy(u_idx).to(dX.device)])
    assert_product("grad_rows", Gg, G, aG, counts.astype(np.float64)[:, None] + 1, None, t)
    if lr and E0 is not None:
        us = 2.0 ** -8 if cfg.dtype == "bf16" else 2.0 ** -24
        E0 = np.asarray(E0, np.float64)
        ref = E0 - lr * Gg                      # on the accelerator's own G
        got = np.asarray(E1, np.float64)
        bound = 2 * us * np.abs(ref) + 4 * 2.0 ** -24 * (np.abs(E0) + abs(lr) * np.abs(Gg))
        flips = int(np.count_nonzero(got != ostep.rounding(cfg.dtype)(ref)))
        print(f"  updated rows [stage]: {flips} of {got.size} elements rounded the other way", flush=True)
        assert np.all(np.abs(got - ref) <= bound + 1e-37)


def to_dev(x, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(x))
    if dtype is not None:
        t = t.to(dtype)
    return t.to(DEV)


def stack_dev(layers, sdt):
    """Stack parameters (numpy, from synth) on the device with zeroed gradients."""
    out = []
    for lay in layers:
        def z(x):
            return torch.zeros(x.shape, dtype=torch.float32, device=DEV)
        d = dict(W=to_dev(lay["W"], sdt), A=to_dev(lay["A"], sdt), gamma=to_dev(lay["gamma"]),
                 C=to_dev(lay["C"], sdt) if lay["C"] is not None else None)
        d.update(dW=z(lay["W"]), dA=z(lay["A"]), dgamma=z(lay["gamma"]),
                 dC=z(lay["C"]) if lay["C"] is not None else None)
        if lay.get("L") is not None:
            d.update(L=to_dev(lay["L"], sdt), dL=z(lay["L"]))
        out.append(d)
    return out


class Workload:
    """Seeded inputs of a config on the GPU, plus the same values for the oracle."""

    def __init__(self, cfg, batch_id=0, tables=None):
        self.cfg = cfg
        sdt = synth.torch_dtype(cfg.dtype)
        self.batch = synth.make_batch(cfg, batch_id)
        self.params = synth.make_dense_params(cfg)
        self.E = synth.make_tables(cfg, device=DEV) if tables is None else tables
        b = self.batch
        self.offsets = to_dev(b["offsets"])
        self.indices = to_dev(b["indices"])
        self.row_base = to_dev(b["row_base"])
        self.dense = to_dev(b["dense"], sdt)
        self.labels = to_dev(b["labels"])
        self.mask = to_dev(b["mask"])
        self.nnz = int(b["offsets"][-1])

        def lin(W, bb):
            return dict(W=to_dev(W, sdt), b=to_dev(bb),
                        dW=torch.zeros(W.shape, dtype=torch.float32, device=DEV),
                        db=torch.zeros(bb.shape, dtype=torch.float32, device=DEV))

        self.bottom = [lin(W, bb) for W, bb in self.params["bottom"]]
        self.top = [lin(W, bb) for W, bb in self.params["top"]]
        for L, (ga, gb) in zip(self.top, self.params.get("top_gain", [])):
            # [2, out], or [D, 2, out] for an untied layer
            L["gain"] = to_dev(np.stack([ga, gb], axis=-2))
            L["dgain"] = torch.zeros(L["gain"].shape, dtype=torch.float32, device=DEV)
        self.domain_offsets = self.batch["domain_offsets"] if cfg.untie else None
        self.fm_W = to_dev(self.params["fm_W"], sdt) if "fm_W" in self.params else None
        self.fm_dW = torch.zeros(self.fm_W.shape, dtype=torch.float32, device=DEV) \
            if self.fm_W is not None else None
        self.stack = stack_dev(self.params["stack"], sdt) if "stack" in self.params else None

    def table_np(self):
        return self.E.float().cpu().double().numpy()

    def step_model(self):
        from paper_2512_09200_amd import api
        c = self.cfg
        return api.StepModel(tables=self.E, row_base=self.row_base, num_features=c.F,
                             dense_in=c.dense_in, bottom=self.bottom, top=self.top,
                             interact=c.interact, fm_W=self.fm_W, fm_dW=self.fm_dW, pool=c.pool,
                             stack=self.stack, stack_n=c.stack_n, ln_eps=c.ln_eps,
                             top_act=c.top_act, norm_block=c.norm_block, norm_eps=c.norm_eps,
                             towers=bool(c.towers), n_domains=len(c.domains[0]) if c.untie else 0,
                             untied_layers=c.untie,
                             skip_absent=c.interact == "dot" and c.domains is not None,
                             fp8_proj=c.stack_fp8)


def relu_overrides(cfg, params, table, batch, gpu_in, gpu_out, max_iter=4):
    """ReLU decisions that the GPU may legitimately take the other way.

    A decision is ambiguous when the float64 pre-activation ``a`` lies within
    ``band = fp32 accumulation bound + |h_gpu - h_ref| @ |W|^T`` of zero: the
    first term covers summation order in fp32, the second the observed
    differences of the layer's (bf16-stored) inputs, which are themselves
    checked against the oracle by the caller.  There the GPU's decision is
    accepted after checking its value is consistent with a pre-activation that
    small; everywhere else the oracle decides.  Iterates until the set is
    stable.  gpu_in / gpu_out: dict "bottom"/"top" -> per-layer input / output
    tensors (None where absent).  Returns (overrides, n_band, n_flipped)."""
    overrides = None
    for _ in range(max_iter):
        c = ostep.forward(cfg, params, table, batch, overrides)
        new, n_band, n_flip = {}, 0, 0
        for name, hs_key, mk, layers in (("bottom", "hs_bottom", "masks_bottom", params["bottom"]),
                                          ("top", "hs_top", "masks_top", params["top"])):
            if hs_key not in c:
                continue
            hs = c[hs_key]
            ov = []
            for i, (W, b) in enumerate(layers):
                out_t = gpu_out[name][i] if i < len(gpu_out[name]) else None
                in_t = gpu_in[name][i] if i < len(gpu_in[name]) else None
                if out_t is None or c[mk][i] is None:
                    ov.append(None)
                    continue
                h_ref = hs[i]
                a = omlp.linear(h_ref, W, b)
                band = omlp.relu_band(h_ref, W, b)
                if in_t is not None:
                    h_gpu = in_t.float().cpu().double().numpy()
                    band = band + np.abs(h_gpu - h_ref) @ np.abs(np.asarray(W, np.float64)).T
                where = np.abs(a) <= band
                g = out_t.float().cpu().double().numpy()
                assert np.all(np.abs(g[where]) <= 2.01 * band[where] + 1e-30), f"{name}{i}: GPU value outside band"
                pos = g > 0
                n_band += int(where.sum())
                n_flip += int((where & (pos != (a > 0))).sum())
                ov.append((where, pos))
            new[name] = ov
        same = overrides is not None and all(
            (x is None and y is None) or (x is not None and y is not None and np.array_equal(x[0], y[0])
                                          and np.array_equal(x[1], y[1]))
            for k in new for x, y in zip(new[k], overrides[k]))
        overrides = new
        if same:
            break
    return overrides, n_band, n_flip
