"""Full-size parity at the workloads' real sizes, in the launch configuration
the benchmark times.  Large embedding (B=8192, 64 tables of 2,000,000 x 128
bf16, ~10.5M lookups): pooled bags, bookkeeping, row gradients and SGD; the
mid workload: the whole step against the oracle; large embedding,
multi-domain (96 tables of 1,000,000 x 128) and deep stack (256 tables of
500,000 x 128, three FM layers): per-sample checks of the whole step.  The
integer bookkeeping is compared in full, bit-exact."""
import numpy as np
import pytest
import torch

import synth
from oracle import embbag as oe
from oracle.bf16 import round_bf16
from tests._util import DEV, assert_close

CFG = synth.LARGE_FM


@pytest.fixture(scope="module")
def big():
    cfg = CFG
    print(f"[fullsize] generating {cfg.name}", flush=True)
    b = synth.make_batch(cfg, 0)
    E = synth.make_tables(cfg, device=DEV)
    d = dict(cfg=cfg, b=b, E=E, offsets=torch.from_numpy(b["offsets"]).to(DEV),
             indices=torch.from_numpy(b["indices"]).to(DEV),
             row_base=torch.from_numpy(b["row_base"]).to(DEV), nnz=int(b["offsets"][-1]))
    torch.cuda.synchronize()
    yield d
    del d["E"]
    torch.cuda.empty_cache()


def _rows(E, rows):
    return E[torch.from_numpy(np.asarray(rows, np.int64)).to(DEV)].float().cpu().double().numpy()


@pytest.mark.gpu
def test_fullsize_embbag_fwd_sampled_bags(big):
    from paper_2512_09200_amd import api
    cfg, b = big["cfg"], big["b"]
    X = torch.empty((cfg.B, cfg.n_slots, cfg.d), dtype=torch.bfloat16, device=DEV)
    api.lattice_embbag_fwd(big["E"], big["row_base"], big["offsets"], big["indices"], cfg.F, cfg.B, X, 1)
    torch.cuda.synchronize()
    r = np.random.default_rng(0)
    bags = np.concatenate([r.choice(cfg.F * cfg.B, 500, replace=False), [0, cfg.F * cfg.B - 1]])
    off = b["offsets"].astype(np.int64)
    got, ref = [], []
    for bag in bags:
        f, s = divmod(int(bag), cfg.B)
        idx = b["indices"][off[bag]:off[bag + 1]].astype(np.int64) + f * cfg.rows
        ref.append(round_bf16(_rows(big["E"], idx).sum(0)))
        got.append(X[s, 1 + f].float().cpu().numpy())
    assert_close("sampled pooled rows", np.array(got), np.array(ref), 2e-2)


@pytest.mark.gpu
def test_fullsize_embbag_bwd_bookkeeping_and_sgd(big):
    from paper_2512_09200_amd import api
    cfg, b = big["cfg"], big["b"]
    print("[fullsize] oracle bookkeeping over all occurrences", flush=True)
    bk = oe.bookkeeping(b["row_base"], b["offsets"], b["indices"], cfg.F, cfg.B)
    uniq, counts, seg = bk["unique_rows"], bk["counts"], bk["seg_offsets"]
    r = np.random.default_rng(1)
    sample_u = np.unique(np.concatenate([r.choice(uniq.size, 300, replace=False),
                                         np.argsort(counts)[-5:], [0, uniq.size - 1]]))
    rows = uniq[sample_u]
    untouched = r.integers(0, cfg.F * cfg.rows, 2000)
    untouched = untouched[~np.isin(untouched, uniq)][:300]
    E_before, E_untouched = _rows(big["E"], rows), _rows(big["E"], untouched)
    dX_np = synth.randn((cfg.B, cfg.n_slots, cfg.d), seed=cfg.seed, stream=7, scale=1e-2, dtype="bf16")
    dX = torch.from_numpy(dX_np).to(torch.bfloat16).to(DEV)
    lr = 50.0  # large enough that the update moves bf16 values
    print("[fullsize] GPU backward", flush=True)
    out = api.lattice_embbag_bwd(big["E"], big["row_base"], big["offsets"], big["indices"], cfg.F,
                                 cfg.B, dX, 1, lr=lr)
    torch.cuda.synchronize()
    U = int(out["num_unique"].item())
    print(f"[fullsize] num_unique GPU {U} oracle {uniq.size}", flush=True)
    assert U == uniq.size
    np.testing.assert_array_equal(out["unique_rows"][:U].cpu().numpy(), uniq)
    np.testing.assert_array_equal(out["seg_offsets"][:U + 1].cpu().numpy(), np.append(seg, big["nnz"]))
    np.testing.assert_array_equal(out["sorted_bags"][:big["nnz"]].cpu().numpy(), bk["sorted_bags"])
    # row gradients of the sampled rows, each summed over its own occurrences
    G = np.zeros((sample_u.size, cfg.d))
    for i, u in enumerate(sample_u):
        bags = bk["sorted_bags"][seg[u]: seg[u] + counts[u]]
        f, s = bags // cfg.B, bags % cfg.B
        G[i] = dX_np[s, 1 + f].astype(np.float64).sum(0)
    assert_close("sampled grad_rows", out["grad_rows"][torch.from_numpy(sample_u).to(DEV)], G, 2e-2)
    assert_close("sampled updated rows", _rows(big["E"], rows), oe.sgd_rows(E_before, G, lr, round_bf16), 2e-2)
    assert np.array_equal(_rows(big["E"], untouched), E_untouched), "untouched rows changed"


@pytest.mark.gpu
def test_fullsize_mid_workload_whole_batch():
    """The mid workload (B=2048, 26 tables of 100,000 x 64 bf16, DOT over 27
    vectors) is small enough for the oracle to recompute the whole step: every
    tensor, every parameter gradient and all row gradients are compared."""
    from tests.test_gpu_step import check_step
    print("[fullsize] mid-dot-bf16 whole batch", flush=True)
    check_step(synth.MID, 0.0)


SAMPLED = {"large-emb-fm": synth.LARGE_FM, "multidomain-dot": synth.MULTIDOMAIN,
           "deep-stack": synth.DEEP_STACK}


@pytest.mark.gpu
@pytest.mark.parametrize("name", list(SAMPLED))
def test_fullsize_step(name):
    """lattice_step at a workload's full size as the benchmark runs it (with
    its SGD step, if any).  (1) Full bookkeeping bit-exact.  (2) Every stage
    recomputed by the oracle from the accelerator's own stored inputs over the
    whole batch: MLP forward and gradient chain, every dense weight and bias
    gradient (top, bottom, FM), the interaction forward / backward, and
    sampled row gradients and SGD updates; for the deep stack (16384
    samples) the per-sample stages on sampled samples and sampled output rows
    of the two largest weight gradients.  (3) The composed step per sample:
    forward and backward outputs and the row gradients (and SGD updates) of
    cold rows, recomputed by the oracle on the samples involved (with the full
    batch's loss normaliser), within the element-wise tolerance or the derived
    deviation."""
    from oracle import bounds as obounds
    from oracle import step as ostep
    from paper_2512_09200_amd import api
    from tests._util import (Workload, assert_close_derived, check_sparse_stage, check_stages, grads_of,
                             relu_overrides)
    cfg = SAMPLED[name]
    lr = cfg.lr_tables
    print(f"[fullsize-step] {name}: generating inputs", flush=True)
    w = Workload(cfg)
    b = w.batch
    model = api.StepModel(tables=w.E, row_base=w.row_base, num_features=cfg.F, dense_in=cfg.dense_in,
                          bottom=w.bottom, top=w.top, interact=cfg.interact, fm_W=w.fm_W,
                          fm_dW=w.fm_dW, pool=cfg.pool, stack=w.stack, stack_n=cfg.stack_n,
                          ln_eps=cfg.ln_eps, max_rows=cfg.rows,
                          skip_absent=cfg.interact == "dot" and cfg.domains is not None)
    print("[fullsize-step] oracle bookkeeping", flush=True)
    bk = oe.bookkeeping(b["row_base"], b["offsets"], b["indices"], cfg.F, cfg.B)
    uniq, counts, seg = bk["unique_rows"], bk["counts"], bk["seg_offsets"]
    r = np.random.default_rng(2)
    cold_u = r.choice(np.flatnonzero(counts <= 2), 40, replace=False)
    sample_u = np.unique(np.concatenate([r.choice(uniq.size, 3000, replace=False), cold_u,
                                         np.argsort(counts)[-20:], [0, uniq.size - 1]]))
    occ_bags = np.concatenate([bk["sorted_bags"][seg[u]: seg[u] + counts[u]] for u in cold_u])
    probe = r.choice(cfg.B, 6, replace=False)
    samples = np.unique(np.concatenate([probe, occ_bags % cfg.B]))
    E_sample_before = _rows(w.E, uniq[sample_u])
    untouched = r.integers(0, cfg.F * cfg.rows, 4000)
    untouched = untouched[~np.isin(untouched, uniq)][:500]
    E_untouched = _rows(w.E, untouched)
    # the oracle's inputs for the composed check: the involved samples and
    # their table rows before the step
    scfg, sub, grows = synth.sub_batch(cfg, b, samples)
    table = _rows(w.E, grows)
    pos = {int(gr): i for i, gr in enumerate(grows)}
    lay = api.lattice_step_plan(model, cfg.B, w.nnz, lr, True)
    ws = torch.zeros(lay.total_bytes, dtype=torch.uint8, device=DEV)
    print(f"[fullsize-step] workspace {lay.total_bytes / 2**30:.2f} GiB", flush=True)
    api.lattice_step(model, w.offsets, w.indices, w.dense, w.labels, w.mask, ws, lr, True,
                     side=api.SideStream())
    torch.cuda.synchronize()
    v = api.step_views(model, ws, lay, cfg.B, cfg.T, w.nnz)

    print("[fullsize-step] stages on the accelerator's own inputs", flush=True)
    big = cfg.B > 8192
    rows = r.choice(cfg.B, 64, replace=False) if big else None
    wrows = ({("top", 0): r.choice(cfg.top[0], 64, replace=False)} if big else None)
    check_stages(cfg, w.params, b, v, grads_of(w), rows=rows, wgrad_rows=wrows)
    check_sparse_stage(cfg, b, v, w.nnz, E_sample_before if lr else None,
                       _rows(w.E, uniq[sample_u]) if lr else None, lr, sample=sample_u, bk=bk)
    assert np.array_equal(_rows(w.E, untouched), E_untouched), "untouched rows changed"

    print(f"[fullsize-step] composed step on {samples.size} samples", flush=True)
    sel = torch.from_numpy(samples).to(DEV)
    gin = dict(bottom=([w.dense[sel]] + [a[sel] for a in v["bottom_act"]]) if cfg.has_dense else [],
               top=[v["t"][sel, :cfg.top_in]] + [a[sel] for a in v["top_act"]])
    gout = dict(bottom=([a[sel] for a in v["bottom_act"]] + [v["X"][sel, 0]]) if cfg.has_dense else [],
                top=[a[sel] for a in v["top_act"]])
    N = float(b["mask"].sum())
    ov, nb, nf = relu_overrides(scfg, w.params, table, sub, gin, gout)
    c, g = ostep.step(scfg, w.params, table, sub, lr_tables=0.0, overrides=ov, loss_normalizer=N)
    bd = obounds.step_bounds(scfg, w.params, table, sub, c, g, lr_tables=0.0, loss_normalizer=N)
    print(f"  ReLU band {nb}, taken the other way {nf}", flush=True)
    s0 = cfg.first_emb_slot
    assert_close("X[emb] (sampled)", v["X"][sel, s0:], c["X"][:, s0:], 2e-2)
    for nm, got, ref, e in [("X", v["X"][sel], c["X"], bd["X"]),
                            ("t", v["t"][sel, :cfg.top_in], c["t"], bd["t"]),
                            ("logits", v["logits"][sel], c["logits"], bd["logits"]),
                            ("d_logits", v["d_logits"][sel], c["dz"], bd["dz"]),
                            ("d_t", v["d_t"][sel, :cfg.top_in], g["d_top_in"], bd["d_top_in"]),
                            ("dX_emb", v["dX"][sel, s0:], g["dX_emb"], bd["dX_emb"])]:
        assert_close_derived(nm + " (sampled)", got, ref, e, 2e-2)
    # cold rows: every occurrence's sample is in the sub-batch, so the oracle's G is exact
    ci = np.array([np.searchsorted(g["unique_rows"], pos[int(uniq[u])]) for u in cold_u])
    assert_close_derived("cold grad_rows", v["grad_rows"][torch.from_numpy(cold_u).to(DEV)],
                         g["grad_rows"][ci], (bd["grad_rows"][0][ci], bd["grad_rows"][1][ci]), 2e-2)
    del w, ws
    torch.cuda.empty_cache()
