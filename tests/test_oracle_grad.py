"""Central finite differences of the oracle's loss against its analytic
gradients, in float64 (no storage rounding), on tiny models with the
structure of each workload: dot interaction with dense path (sum and mean
pooling), FM block, and the stacked FM -> linear -> residual -> LayerNorm
block (with a compression residual on its first layer).  Masks include
zeros, so masked heads are covered."""
import numpy as np
import pytest

import synth
from oracle import interact, mlp, step, swishrn


def _tiny_cfg(kind, pool="sum"):
    base = dict(B=5, rows=4, d=4, dtype="f32", index_dist=("uniform",),
                bag_dist=("uniform", 0, 3), label_p=("fixed", 0.4), mask=("iid", 0.6),
                pool=pool, seed=1234)
    if kind == "dot":
        return synth.Config(name="t-dot", F=3, dense_in=3, bottom=(6, 4), interact="dot",
                            top=(5, 3), **base)
    if kind == "fm":
        return synth.Config(name="t-fm", F=3, dense_in=3, bottom=(5, 4), interact="fm",
                            fm_rank=2, top=(6, 3), **base)
    if kind == "stack":
        return synth.Config(name="t-stack", F=5, dense_in=0, bottom=(), interact="stack",
                            fm_rank=2, stack_layers=2, stack_n=3, top=(4, 2), **base)
    if kind == "untied":
        # two domains (seeded sizes), the first two top layers untied, SwishRN
        return synth.Config(name="t-untied", F=4, dense_in=3, bottom=(6, 4), interact="dot",
                            top=(5, 6, 3), untie=2, top_act="swishrn", norm_block=2, norm_eps=1e-3,
                            domains=((0.6, 0.4), 3, 2), **dict(base, mask=("domain",)))
    if kind == "towers":
        # per-objective towers: 3 objectives x 2 hidden units, then grouped heads
        return synth.Config(name="t-towers", F=3, dense_in=3, bottom=(6, 4), interact="dot",
                            top=(5, 6, 3), towers=2, **base)
    if kind == "dwfb":
        # full fusion blocks: 2 of the 3 output vectors from the FM block, 1 from
        # the linear compression block
        return synth.Config(name="t-dwfb", F=5, dense_in=0, bottom=(), interact="stack",
                            fm_rank=2, stack_layers=2, stack_n=3, lcb_n=1, top=(4, 2), **base)
    if kind in ("swishrn", "hardswishrn"):
        # SwishRN hidden top layers, BlockNorm groups of 2 (3, 2, 2, 1 features
        # over widths 7 and 5: a ragged last group)
        return synth.Config(name="t-" + kind, F=3, dense_in=3, bottom=(6, 4), interact="dot",
                            top=(7, 5, 3), top_act=kind, norm_block=2, norm_eps=1e-3, **base)
    raise ValueError(kind)


def _setup(cfg):
    batch = synth.make_batch(cfg)
    p = synth.make_dense_params(cfg)
    # float64 copies so perturbations are not lost to fp32 storage
    params = {
        "bottom": [(W.astype(np.float64), b.astype(np.float64)) for W, b in p["bottom"]],
        "top": [(W.astype(np.float64), b.astype(np.float64)) for W, b in p["top"]],
    }
    if "fm_W" in p:
        params["fm_W"] = p["fm_W"].astype(np.float64)
    if "top_gain" in p:
        params["top_gain"] = [(ga.astype(np.float64), gb.astype(np.float64)) for ga, gb in p["top_gain"]]
    if "stack" in p:
        params["stack"] = [{k: (None if v is None else v.astype(np.float64)) for k, v in lay.items()}
                           for lay in p["stack"]]
    table = synth.make_tables(cfg).double().numpy().copy()
    return batch, params, table


def _pairs(cfg, params, g):
    """(parameter array, its analytic gradient, name)."""
    out = []
    for i, (W, b) in enumerate(params["bottom"]):
        out += [(W, g["bottom_dW"][i], f"bottom{i}.W"), (b, g["bottom_db"][i], f"bottom{i}.b")]
    for i, (W, b) in enumerate(params["top"]):
        out += [(W, g["top_dW"][i], f"top{i}.W"), (b, g["top_db"][i], f"top{i}.b")]
    if "fm_W" in params:
        out.append((params["fm_W"], g["fm_dW"], "fm.W"))
    for i, (ga, gb) in enumerate(params.get("top_gain", [])):
        out += [(ga, g["top_dgain"][i][0], f"top{i}.ga"), (gb, g["top_dgain"][i][1], f"top{i}.gb")]
    for i, lay in enumerate(params.get("stack", [])):
        sg = g["stack"][i]
        out += [(lay["W"], sg["dW"], f"stack{i}.W"), (lay["A"], sg["dA"], f"stack{i}.A"),
                (lay["gamma"], sg["dgamma"], f"stack{i}.gamma")]
        if lay.get("L") is not None:
            out.append((lay["L"], sg["dL"], f"stack{i}.L"))
        if lay["C"] is not None:
            out.append((lay["C"], sg["dC"], f"stack{i}.C"))
    return out


def _fd(loss_fn, arr, idx, h):
    old = arr[idx]
    arr[idx] = old + h
    lp = loss_fn()
    arr[idx] = old - h
    lm = loss_fn()
    arr[idx] = old
    return (lp - lm) / (2 * h)


def _check_kinks(cfg, params, table, batch):
    """The FD test is only meaningful away from ReLU kinks (and the hard
    gate's kinks at +-3)."""
    c = step.forward(cfg, params, table, batch)
    act = step.top_act(cfg, params)
    for hs, layers, top in ((c.get("hs_bottom"), params["bottom"], False), (c["hs_top"], params["top"], True)):
        if hs is None:
            continue
        for i, (W, b) in enumerate(layers):
            if top and i == len(layers) - 1:
                continue                                   # the heads are linear
            a = mlp.untied_linear(hs[i], W, b, batch["domain"]) if np.ndim(W) == 3 else hs[i] @ W.T + b
            if top and act is not None and i < len(layers) - 1:
                if act["kind"] == "hard":
                    assert np.ndim(act["gains"][i][0]) == 1, "hard-gate kink check: tied gains only"
                    _, n, _ = swishrn.forward(a, *act["gains"][i], act["block"], act["eps"], "hard")
                    z = act["gains"][i][1] * n
                    assert np.min(np.abs(np.abs(z) - 3.0)) > 1e-4, "seed puts a gate input on a kink"
                continue
            assert np.min(np.abs(a)) > 1e-4, "seed puts a pre-activation on a ReLU kink"


def _fd_worst(kind, pool="sum", n_coords=12):
    """Largest relative disagreement between the oracle's analytic gradients
    and central finite differences of its loss, over sampled coordinates of
    every parameter and every touched table row."""
    cfg = _tiny_cfg(kind, pool)
    batch, params, table = _setup(cfg)
    assert batch["mask"].min() == 0 and batch["mask"].max() == 1
    assert (np.diff(batch["offsets"]) == 0).any()           # includes empty bags
    _check_kinks(cfg, params, table, batch)
    c, g = step.step(cfg, params, table, batch, lr_tables=0.0)

    def loss_fn():
        return step.forward(cfg, params, table, batch)["loss"]

    rng = np.random.default_rng(7)
    worst = 0.0
    for arr, grad, name in _pairs(cfg, params, g):
        assert grad.shape == arr.shape, name
        scale = max(np.sqrt(np.mean(grad ** 2)), 1e-12)
        flat = [np.unravel_index(k, arr.shape) for k in
                rng.choice(arr.size, size=min(arr.size, n_coords), replace=False)]
        for idx in flat:
            h = 1e-6 * max(1.0, abs(arr[idx]))
            fd = _fd(loss_fn, arr, idx, h)
            worst = max(worst, abs(fd - grad[idx]) / max(abs(grad[idx]), scale))
    # embedding gradient: every touched row, a few coordinates
    uniq, G = g["unique_rows"], g["grad_rows"]
    scale = max(np.sqrt(np.mean(G ** 2)), 1e-12)
    for u, r in enumerate(uniq):
        for a in rng.choice(cfg.d, size=2, replace=False):
            fd = _fd(loss_fn, table, (r, a), 1e-6)
            worst = max(worst, abs(fd - G[u, a]) / max(abs(G[u, a]), scale))
    # rows that no bag touches have no gradient: perturbing them leaves the loss unchanged
    untouched = np.setdiff1d(np.arange(table.shape[0]), uniq)
    if untouched.size:
        assert _fd(loss_fn, table, (int(untouched[0]), 0), 1e-3) == 0.0
    return worst


@pytest.mark.parametrize("kind,pool", [("dot", "sum"), ("dot", "mean"), ("fm", "sum"), ("stack", "sum"),
                                       ("dwfb", "sum"), ("towers", "sum"), ("untied", "sum"), ("swishrn", "sum"),
                                       ("hardswishrn", "sum")])
def test_finite_differences(kind, pool):
    assert _fd_worst(kind, pool) < 1e-6


# ------------------------------------------------------------------------
# Planted mistakes: each copy of a backward function below carries one
# plausible error; the finite-difference pin must catch it.
def _fm_backward_wrong_sign(G, X, W, P, rnd):
    G, X, W = (np.asarray(a, np.float64) for a in (G, X, W))
    dP = rnd(X.transpose(0, 2, 1) @ G)
    dX = G @ P.transpose(0, 2, 1) - W[None] @ dP.transpose(0, 2, 1)     # sign of the W term
    return dX, (X @ dP).sum(axis=0)


def _layernorm_backward_dropped_term(dy, xhat, rstd, gamma):
    dy = np.asarray(dy, np.float64)
    dgamma = (dy * xhat).reshape(-1, xhat.shape[-1]).sum(axis=0)
    dxh = dy * np.asarray(gamma, np.float64)
    du = rstd * (dxh - dxh.mean(axis=-1, keepdims=True))              # xhat term dropped
    return du, dgamma


def _mlp_backward_no_relu_mask(g_out, hs, masks, layers, rnd, relu_last, need_input_grad, **kw):
    masks = [None if m is None else np.ones_like(m) for m in masks]
    return _ORIG["mlp_backward"](g_out, hs, masks, layers, rnd, relu_last, need_input_grad, **kw)


def _grouped_grads_wrong_tower(g, h, W):
    dW, db, dh = _ORIG["grouped_linear_grads"](g, h, W)
    T, H = W.shape
    return dW, db, dh.reshape(-1, T, H)[:, ::-1].reshape(-1, T * H)      # gradient sent to the wrong tower


def _untied_grads_swapped_sets(g, h, W, domain):
    dW, db, dh = _ORIG["untied_linear_grads"](g, h, W, domain)
    return dW[::-1].copy(), db[::-1].copy(), dh                      # each domain's gradient to the other set


def _swishrn_backward_no_mean_term(do, h, ga, gb, block, eps, kind, rho=None, grad_override=None):
    do = np.asarray(do, np.float64)
    _, n, rho = swishrn.forward(h, ga, gb, block, eps, kind, rho)
    a, z = ga * n, gb * n
    s, sp = swishrn.gate(z, kind), swishrn.gate_grad(z, kind)
    dn = ga * do * s + gb * do * a * sp
    dh = swishrn.expand(rho, n.shape[1], block) * dn                  # the normalisation's mean term dropped
    return dh, (do * s * n).sum(0), (do * a * sp * n).sum(0)


def _swishrn_backward_whole_row_mean(do, h, ga, gb, block, eps, kind, rho=None, grad_override=None):
    dh, dga, dgb = _ORIG["swishrn_backward"](do, h, ga, gb, block, eps, kind, rho, grad_override)
    _, n, rho = swishrn.forward(h, ga, gb, block, eps, kind, rho)
    a, z = ga * n, gb * n
    dn = ga * do * swishrn.gate(z, kind) + gb * do * a * swishrn.gate_grad(z, kind)
    R = swishrn.expand(rho, n.shape[1], block)
    return R * (dn - n * np.mean(dn * n, axis=1, keepdims=True)), dga, dgb   # mean over the row, not the group


def _swishrn_backward_gate_gain_swapped(do, h, ga, gb, block, eps, kind, rho=None, grad_override=None):
    return _ORIG["swishrn_backward"](do, h, gb, ga, block, eps, kind, rho, grad_override)


def _dot_backward_no_slot0(dp, X):
    dX = _ORIG["dot_backward"](dp, X)
    dX[:, 0] = 0.0                                                    # dense slot's gradient dropped
    return dX


_ORIG = dict(mlp_backward=step.mlp_backward, dot_backward=step.dot_backward,
             swishrn_backward=swishrn.backward, grouped_linear_grads=mlp.grouped_linear_grads,
             untied_linear_grads=mlp.untied_linear_grads)


@pytest.mark.parametrize("target,module,name,kind", [
    (_fm_backward_wrong_sign, step, "fm_backward", "fm"),
    (_layernorm_backward_dropped_term, interact, "layernorm_backward", "stack"),
    (_mlp_backward_no_relu_mask, step, "mlp_backward", "dot"),
    (_dot_backward_no_slot0, step, "dot_backward", "dot"),
    (_swishrn_backward_no_mean_term, swishrn, "backward", "swishrn"),
    (_swishrn_backward_whole_row_mean, swishrn, "backward", "hardswishrn"),
    (_swishrn_backward_gate_gain_swapped, swishrn, "backward", "swishrn"),
    (_grouped_grads_wrong_tower, mlp, "grouped_linear_grads", "towers"),
    (_untied_grads_swapped_sets, mlp, "untied_linear_grads", "untied"),
], ids=["fm-sign", "layernorm-term", "relu-mask", "slot0-gradient", "swishrn-mean-term",
        "blocknorm-group", "swishrn-gains", "tower-routing", "untied-sets"])
def test_planted_backward_mistakes_fail_the_finite_difference_pin(monkeypatch, target, module, name, kind):
    monkeypatch.setattr(module, name, target)
    assert _fd_worst(kind, n_coords=6) > 1e-3
