"""Degenerate inputs of the step and of the pooled lookup, on the GPU:
every label masked, an empty batch, a batch with no lookups, and no
categorical features (Section 3.2.1: an impression trains only its routed
heads, so a batch routed to no head trains nothing; Section 3.2: absent
features are empty bags)."""
import numpy as np
import pytest
import torch

import synth
from oracle import embbag as oe
from oracle import step as ostep
from tests._util import DEV, Workload
from tests.test_gpu_step import check_step, run_step


def _grads(w):
    out = [L[k] for L in w.top + w.bottom for k in ("dW", "db")]
    if w.fm_dW is not None:
        out.append(w.fm_dW)
    for lay in w.stack or []:
        out += [lay[k] for k in ("dW", "dA", "dgamma", "dC") if lay.get(k) is not None]
    return out


def _poison(w):
    for g in _grads(w):
        g.fill_(float("nan"))


@pytest.mark.gpu
@pytest.mark.parametrize("name", ["large-fm", "mid", "deep-stack"])
def test_all_labels_masked_trains_nothing(name):
    """N = max(1, sum m) = 1, so L = 0 and dz = 0 exactly; every gradient is
    then exactly zero and the SGD step leaves the tables bit-identical."""
    cfg = {"large-fm": synth.small(synth.LARGE_FM, B=96, rows=3000),
           "mid": synth.small(synth.MID, B=200, rows=3000),
           "deep-stack": synth.DEEP_STACK.scaled(B=40, F=24, rows=800, d=64, stack_n=8, fm_rank=16,
                                                top=(128, 32, 8))}[name]
    print(f"[edge] all-masked {name} B={cfg.B}", flush=True)
    w = Workload(cfg)
    w.mask.zero_()
    w.batch["mask"][:] = 0
    E0 = w.E.clone()
    _poison(w)
    _, v, _ = run_step(w, 0.05)
    c, _ = ostep.step(cfg, w.params, w.table_np(), w.batch, lr_tables=0.05)
    assert c["loss"] == 0.0 and not np.any(c["dz"])          # the oracle agrees
    assert v["loss"].item() == 0.0
    assert torch.count_nonzero(v["d_logits"]) == 0
    assert torch.count_nonzero(v["dX"]) == 0
    U = int(v["num_unique"].item())
    assert U == np.unique(oe.row_keys(w.batch["row_base"], w.batch["offsets"],
                                                 w.batch["indices"], cfg.F, cfg.B)).size
    assert torch.count_nonzero(v["grad_rows"][:U]) == 0
    for g in _grads(w):
        assert torch.count_nonzero(g) == 0
    assert torch.equal(w.E, E0)


@pytest.mark.gpu
def test_empty_batch_zeroes_the_gradients():
    """B = 0: every parameter gradient is a sum over no samples, so it is
    written as zero; the loss and the unique-row count are zero; the tables
    are untouched."""
    from paper_2512_09200_amd import api
    cfg = synth.small(synth.LARGE_FM, B=64, rows=2000)
    w = Workload(cfg)
    model = w.step_model()
    lay = api.lattice_step_plan(model, 0, 0, 0.05, True)
    ws = torch.full((max(lay.total_bytes, 1),), 0x7f, dtype=torch.uint8, device=DEV)
    E0 = w.E.clone()
    _poison(w)
    empty_i = torch.zeros(0, dtype=torch.int32, device=DEV)
    api.lattice_step(model, torch.zeros(1, dtype=torch.int32, device=DEV), empty_i,
                     torch.zeros((0, cfg.dense_in), dtype=w.dense.dtype, device=DEV),
                     torch.zeros((0, cfg.T), device=DEV), torch.zeros((0, cfg.T), dtype=torch.uint8, device=DEV),
                     ws, 0.05, True, side=api.SideStream())
    torch.cuda.synchronize()
    v = api.step_views(model, ws, lay, 0, cfg.T, 0)
    assert v["loss"].item() == 0.0 and int(v["num_unique"].item()) == 0
    for g in _grads(w):
        assert torch.count_nonzero(g) == 0
    assert torch.equal(w.E, E0)


@pytest.mark.gpu
@pytest.mark.parametrize("name", ["large-fm", "mid"])
def test_batch_without_lookups_matches_oracle(name):
    """nnz = 0 with B > 0: every bag is empty, so every embedding slot pools
    to zero, nothing occurs in the sparse gradient and no table row moves;
    the dense path still trains and matches the oracle."""
    cfg = {"large-fm": synth.small(synth.LARGE_FM, B=96, rows=3000),
           "mid": synth.small(synth.MID, B=160, rows=3000)}[name]
    print(f"[edge] nnz=0 {name} B={cfg.B}", flush=True)
    w = Workload(cfg)
    w.batch["offsets"] = np.zeros_like(w.batch["offsets"])
    w.batch["indices"] = w.batch["indices"][:0]
    w.offsets = torch.zeros_like(w.offsets)
    w.indices = w.indices[:0]
    w.nnz = 0
    check_step(cfg, 0.05, w=w)


@pytest.mark.gpu
def test_no_features_is_a_noop_for_the_lookup_and_rejected_by_the_step():
    """F = 0: the pooled lookup writes nothing and its gradient has no rows;
    the step needs at least one categorical feature and says so."""
    from paper_2512_09200_amd import api
    from paper_2512_09200_amd._abi import LatticeError
    E = torch.randn(100, 64, device=DEV).to(torch.bfloat16)
    row_base = torch.zeros(1, dtype=torch.int64, device=DEV)
    offsets = torch.zeros(1, dtype=torch.int32, device=DEV)
    indices = torch.zeros(0, dtype=torch.int32, device=DEV)
    X = torch.full((8, 1, 64), 3.0, device=DEV).to(torch.bfloat16)
    api.lattice_embbag_fwd(E, row_base, offsets, indices, 0, 8, X, first_slot=1)
    torch.cuda.synchronize()
    assert torch.all(X == 3.0)
    out = api.lattice_embbag_bwd(E, row_base, offsets, indices, 0, 8, X, first_slot=1)
    torch.cuda.synchronize()
    assert int(out["num_unique"].item()) == 0
    cfg = synth.small(synth.MID, B=16, rows=100)
    w = Workload(cfg)
    m = w.step_model()
    m.desc.num_features = 0
    with pytest.raises(LatticeError, match="INVALID_ARG"):
        api.lattice_step_plan(m, cfg.B, 0)
