"""Pins of parameter untying (Section 3.3.4): a domain's samples use only
its own parameter set, so (a) with every set equal the untied step is the
tied step, and (b) changing one domain's set changes exactly that domain's
samples."""
import numpy as np

import synth
from oracle import step


def _cfg():
    return synth.small(synth.MULTIDOMAIN, B=48, rows=200, F=12, top=(32, 16, 6),
                       domains=((0.5, 0.3, 0.2), 8, 3), untie=2)


def _setup(cfg):
    batch = synth.make_batch(cfg)
    params = synth.make_dense_params(cfg)
    table = synth.make_tables(cfg).double().numpy()
    return batch, params, table


def test_equal_sets_are_the_tied_model():
    cfg = _cfg()
    batch, params, table = _setup(cfg)
    assert np.all(np.diff(batch["domain"]) >= 0)           # grouped by domain
    tied = dict(params, top=[(W[0], b[0]) if np.ndim(W) == 3 else (W, b) for W, b in params["top"]])
    same = dict(params, top=[(np.stack([W[0]] * W.shape[0]), np.stack([b[0]] * b.shape[0])) if np.ndim(W) == 3
                             else (W, b) for W, b in params["top"]])
    ct, gt = step.step(cfg.scaled(untie=0), tied, table, batch)
    cu, gu = step.step(cfg, same, table, batch)
    assert np.max(np.abs(ct["logits"] - cu["logits"])) < 1e-12
    assert np.max(np.abs(gt["d_top_in"] - gu["d_top_in"])) < 1e-12
    for i in range(cfg.untie):
        # the tied gradient is the sum of the sets' gradients
        assert np.max(np.abs(gt["top_dW"][i] - gu["top_dW"][i].sum(0))) < 1e-12


def test_a_domain_set_reaches_only_its_samples():
    cfg = _cfg()
    batch, params, table = _setup(cfg)
    c0 = step.forward(cfg, params, table, batch)
    W0, b0 = params["top"][0]
    W1 = W0.copy()
    W1[1] *= 1.5                                            # domain 1's first-layer set only
    c1 = step.forward(cfg, dict(params, top=[(W1, b0)] + params["top"][1:]), table, batch)
    changed = np.any(c1["logits"] != c0["logits"], axis=1)
    assert np.array_equal(changed, batch["domain"] == 1)
    assert changed.any()
    _, g = step.step(cfg, params, table, batch)
    for k in range(W0.shape[0]):
        rows = batch["domain"] == k
        # set k's bias gradient is the sum over its own samples of the layer's pre-activation gradient
        assert np.any(g["top_db"][0][k] != 0) == bool(rows.any())
