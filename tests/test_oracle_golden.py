"""Hand-worked example (tests/golden/worked_dot_example.json) and a sanity
bound between the bf16-storage and float64 modes of the oracle."""
import json
import math
import os

import numpy as np

import synth
from oracle import interact, step
from oracle.bf16 import identity, round_bf16
from oracle.metrics import max_rel_err

HERE = os.path.dirname(os.path.abspath(__file__))


def test_worked_example():
    g = json.load(open(os.path.join(HERE, "golden", "worked_dot_example.json")))
    cfg = synth.Config(name="worked", B=1, F=2, rows=3, d=2, dtype="f32", index_dist=("uniform",),
                       bag_dist=("uniform", 1, 1), dense_in=0, bottom=(), interact="dot", top=(1,),
                       lr_tables=g["lr"])
    batch = dict(offsets=np.array(g["offsets"], np.int32), indices=np.array(g["indices"], np.int32),
                 row_base=np.array([0, 3, 6]), labels=np.array(g["labels"]), mask=np.array(g["mask"]),
                 dense=np.zeros((1, 0)))
    params = dict(bottom=[], top=[(np.array(g["top_W"]), np.array(g["top_b"]))])
    table = np.array(g["tables"], np.float64)
    c, gr = step.step(cfg, params, table, batch)
    e = g["expect"]
    np.testing.assert_array_equal(c["X"], e["pooled"])
    np.testing.assert_array_equal(c["inter"], e["pairs"])
    np.testing.assert_array_equal(c["logits"], e["logits"])
    assert abs(c["loss"] - math.log(2.0)) < 1e-15 and abs(e["loss"] - math.log(2.0)) < 1e-15
    np.testing.assert_array_equal(c["dz"], e["dz"])
    np.testing.assert_array_equal(gr["top_dW"][0], e["top_dW"])
    np.testing.assert_array_equal(gr["top_db"][0], e["top_db"])
    np.testing.assert_array_equal(gr["dX_emb"], e["dX_emb"])
    np.testing.assert_array_equal(gr["unique_rows"], e["unique_rows"])
    np.testing.assert_array_equal(gr["bookkeeping"]["counts"], e["counts"])
    np.testing.assert_array_equal(gr["bookkeeping"]["seg_offsets"], e["seg_offsets"])
    np.testing.assert_array_equal(gr["bookkeeping"]["sorted_positions"], e["sorted_positions"])
    np.testing.assert_array_equal(gr["grad_rows"], e["grad_rows"])
    np.testing.assert_array_equal(gr["updated_rows"], e["updated_rows"])


def test_bf16_storage_mode_stays_close_to_float64_mode():
    # the storage points only perturb values at the bf16 rounding level
    cfg16 = synth.small(synth.MID, B=64, rows=500)
    cfg64 = cfg16.scaled(dtype="f32")
    batch = synth.make_batch(cfg16)
    params = synth.make_dense_params(cfg16)              # bf16-valued weights for both modes
    table = synth.make_tables(cfg16).double().numpy()
    c16, g16 = step.step(cfg16, params, table, batch)
    c64, g64 = step.step(cfg64, params, table, batch)
    assert abs(c16["loss"] - c64["loss"]) < 1e-3 * abs(c64["loss"])
    # norm-wise: a ReLU whose pre-activation sits near zero may flip between
    # the two modes and move single elements by O(1)
    rel = lambda a, b: np.linalg.norm(a - b) / np.linalg.norm(b)
    assert rel(c16["logits"], c64["logits"]) < 0.02
    for i in range(3):
        assert rel(g16["top_dW"][i], g64["top_dW"][i]) < 0.05
    assert rel(g16["bottom_dW"][0], g64["bottom_dW"][0]) < 0.05
    assert rel(g16["grad_rows"], g64["grad_rows"]) < 0.05
    # and they are not identical: rounding does happen in bf16 mode
    assert max_rel_err(c16["logits"], c64["logits"]) > 0


def _rel(a, b):
    return np.linalg.norm(np.asarray(a) - np.asarray(b)) / np.linalg.norm(np.asarray(b))


def test_bf16_storage_mode_stays_close_to_the_unrounded_fm_definition():
    # bf16 mode evaluates the FM block as X (X^T W) with P = X^T W rounded
    # (and dP in the backward); the definition is (X X^T) W, which float64
    # mode evaluates with no rounding (the two associations agree to ~1e-13).
    # The interaction is compared on identical inputs and upstream gradients,
    # so only its own storage points differ.
    cfg = synth.small(synth.LARGE_FM, B=48, rows=400)
    batch = synth.make_batch(cfg)
    params = synth.make_dense_params(cfg)
    table = synth.make_tables(cfg).double().numpy()
    c64, g64 = step.step(cfg.scaled(dtype="f32"), params, table, batch)
    X, W = round_bf16(c64["X"]), params["fm_W"]
    gram_W = np.einsum("bij,jk->bik", X @ X.transpose(0, 2, 1), W)
    O64, P64 = interact.fm_forward(X, W, identity)
    assert _rel(O64, gram_W) < 1e-12
    O16, P16 = interact.fm_forward(X, W, round_bf16)
    assert 0 < _rel(O16, gram_W) < 0.01
    G = round_bf16(g64["d_top_in"][:, cfg.d:].reshape(O64.shape))
    dX64, dW64 = interact.fm_backward(G, X, W, P64, identity)
    dX16, dW16 = interact.fm_backward(G, X, W, P16, round_bf16)
    assert 0 < _rel(dX16, dX64) < 0.01
    assert 0 < _rel(dW16, dW64) < 0.01
    c16, _ = step.step(cfg, params, table, batch)
    assert abs(c16["loss"] - c64["loss"]) < 1e-3 * abs(c64["loss"])


def test_bf16_storage_mode_stays_close_to_float64_mode_for_the_stack():
    cfg = synth.DEEP_STACK.scaled(B=24, F=16, rows=300, d=32, stack_n=8, fm_rank=8, top=(64, 16, 4))
    batch = synth.make_batch(cfg)
    params = synth.make_dense_params(cfg)
    table = synth.make_tables(cfg).double().numpy()
    c64, g64 = step.step(cfg.scaled(dtype="f32"), params, table, batch)
    X = round_bf16(c64["X"])
    Y64, k64 = interact.stack_forward(X, params["stack"], cfg.stack_n, cfg.d, identity, cfg.ln_eps)
    Y16, k16 = interact.stack_forward(X, params["stack"], cfg.stack_n, cfg.d, round_bf16, cfg.ln_eps)
    assert 0 < _rel(Y16, Y64) < 0.02
    dY = round_bf16(g64["d_top_in"].reshape(Y64.shape))
    dX64, s64 = interact.stack_backward(dY, params["stack"], k64, identity)
    dX16, s16 = interact.stack_backward(dY, params["stack"], k16, round_bf16)
    assert 0 < _rel(dX16, dX64) < 0.03
    for l, (a, b) in enumerate(zip(s16, s64)):
        for k in ("dW", "dA", "dgamma"):
            assert _rel(a[k], b[k]) < 0.03, (l, k)
    c16, _ = step.step(cfg, params, table, batch)
    assert abs(c16["loss"] - c64["loss"]) < 1e-3 * abs(c64["loss"])
