"""Central finite differences of the oracle's loss against its analytic
gradients, in float64 (no storage rounding), on tiny models with the
structure of each workload: dot interaction with dense path (sum and mean
pooling), FM block, and the stacked FM -> linear -> residual -> LayerNorm
block (with a compression residual on its first layer).  Masks include
zeros, so masked heads are covered."""
import numpy as np
import pytest

import synth
from oracle import step


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
    for i, lay in enumerate(params.get("stack", [])):
        sg = g["stack"][i]
        out += [(lay["W"], sg["dW"], f"stack{i}.W"), (lay["A"], sg["dA"], f"stack{i}.A"),
                (lay["gamma"], sg["dgamma"], f"stack{i}.gamma")]
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
    """The FD test is only meaningful away from ReLU kinks."""
    c = step.forward(cfg, params, table, batch)
    for hs, layers in ((c.get("hs_bottom"), params["bottom"]), (c["hs_top"], params["top"])):
        if hs is None:
            continue
        for i, (W, b) in enumerate(layers):
            a = hs[i] @ W.T + b
            assert np.min(np.abs(a)) > 1e-4, "seed puts a pre-activation on a ReLU kink"


@pytest.mark.parametrize("kind,pool", [("dot", "sum"), ("dot", "mean"), ("fm", "sum"), ("stack", "sum")])
def test_finite_differences(kind, pool):
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
                rng.choice(arr.size, size=min(arr.size, 12), replace=False)]
        for idx in flat:
            h = 1e-6 * max(1.0, abs(arr[idx]))
            fd = _fd(loss_fn, arr, idx, h)
            err = abs(fd - grad[idx]) / max(abs(grad[idx]), scale)
            worst = max(worst, err)
            assert err < 1e-6, (name, idx, fd, grad[idx])
    # embedding gradient: every touched row, a few coordinates
    uniq, G = g["unique_rows"], g["grad_rows"]
    scale = max(np.sqrt(np.mean(G ** 2)), 1e-12)
    for u, r in enumerate(uniq):
        for a in rng.choice(cfg.d, size=2, replace=False):
            fd = _fd(loss_fn, table, (r, a), 1e-6)
            err = abs(fd - G[u, a]) / max(abs(G[u, a]), scale)
            worst = max(worst, err)
            assert err < 1e-6, ("table", r, a, fd, G[u, a])
    # rows that no bag touches have no gradient: perturbing them leaves the loss unchanged
    untouched = np.setdiff1d(np.arange(table.shape[0]), uniq)
    if untouched.size:
        assert _fd(loss_fn, table, (int(untouched[0]), 0), 1e-3) == 0.0
