"""Full-size parity at the large-embedding workload (B=8192, 64 tables of
2,000,000 x 128 bf16, Zipf 1.05, ~10.5M lookups), in the launch configuration
the benchmark times.  The oracle checks sampled outputs it can compute one by
one (pooled bags, row gradients, updated rows); the integer bookkeeping is
compared in full, bit-exact."""
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


def _dev_params(cfg):
    p = synth.make_dense_params(cfg)
    sdt = synth.torch_dtype(cfg.dtype)

    def lin(W, b):
        return dict(W=torch.from_numpy(W).to(sdt).to(DEV), b=torch.from_numpy(b).to(DEV),
                    dW=torch.zeros(W.shape, device=DEV), db=torch.zeros(b.shape, device=DEV))
    return p, [lin(W, b) for W, b in p["bottom"]], [lin(W, b) for W, b in p["top"]], \
        torch.from_numpy(p["fm_W"]).to(sdt).to(DEV)


@pytest.mark.gpu
def test_fullsize_step_per_sample(big):
    """lattice_step at full size as the benchmark runs it (SGD lr 0.01): full
    bookkeeping bit-exact; per-sample forward/backward outputs and the row
    gradients and SGD updates of cold rows, each recomputed by the oracle on
    the samples involved (with the full batch's loss normaliser)."""
    from oracle import step as ostep
    from paper_2512_09200_amd import api
    from tests._util import assert_close_composed, relu_overrides
    cfg, b = big["cfg"], big["b"]
    params, bottom, top, fm_W = _dev_params(cfg)
    fm_dW = torch.zeros(tuple(fm_W.shape), device=DEV)
    model = api.StepModel(tables=big["E"], row_base=big["row_base"], num_features=cfg.F,
                          dense_in=cfg.dense_in, bottom=bottom, top=top, interact="fm",
                          fm_W=fm_W, fm_dW=fm_dW)
    bk = oe.bookkeeping(b["row_base"], b["offsets"], b["indices"], cfg.F, cfg.B)
    uniq, counts, seg = bk["unique_rows"], bk["counts"], bk["seg_offsets"]
    r = np.random.default_rng(2)
    cold = np.flatnonzero(counts <= 2)
    cold_u = r.choice(cold, 40, replace=False)
    occ_bags = np.concatenate([bk["sorted_bags"][seg[u]: seg[u] + counts[u]] for u in cold_u])
    probe = r.choice(cfg.B, 6, replace=False)
    samples = np.unique(np.concatenate([probe, occ_bags % cfg.B]))
    E_cold_before = _rows(big["E"], uniq[cold_u])
    # the oracle's inputs: the involved samples and their table rows before the step
    scfg, sub, grows = synth.sub_batch(cfg, b, samples)
    table = _rows(big["E"], grows)
    pos = {int(g): i for i, g in enumerate(grows)}
    dense = torch.from_numpy(b["dense"]).to(torch.bfloat16).to(DEV)
    labels, mask = torch.from_numpy(b["labels"]).to(DEV), torch.from_numpy(b["mask"]).to(DEV)
    lay = api.lattice_step_plan(model, cfg.B, big["nnz"], cfg.lr_tables, True)
    ws = torch.zeros(lay.total_bytes, dtype=torch.uint8, device=DEV)
    print(f"[fullsize-step] workspace {lay.total_bytes / 2**30:.2f} GiB; {samples.size} samples checked", flush=True)
    api.lattice_step(model, big["offsets"], big["indices"], dense, labels, mask, ws, cfg.lr_tables, True)
    torch.cuda.synchronize()
    v = api.step_views(model, ws, lay, cfg.B, cfg.T, big["nnz"])
    U = int(v["num_unique"].item())
    print(f"[fullsize-step] num_unique GPU {U} oracle {uniq.size}", flush=True)
    assert U == uniq.size
    np.testing.assert_array_equal(v["unique_rows"][:U].cpu().numpy(), uniq)
    np.testing.assert_array_equal(v["sorted_bags"][:big["nnz"]].cpu().numpy(), bk["sorted_bags"])
    sel = torch.from_numpy(samples).to(DEV)
    gin = dict(bottom=[dense[sel], v["bottom_act"][0][sel]],
               top=[v["t"][sel, :cfg.top_in]] + [a[sel] for a in v["top_act"]])
    gout = dict(bottom=[v["bottom_act"][0][sel], v["X"][sel, 0]], top=[a[sel] for a in v["top_act"]])
    N = float(b["mask"].sum())
    ov, nb, nf = relu_overrides(scfg, params, table, sub, gin, gout)
    c, g = ostep.step(scfg, params, table, sub, lr_tables=0.0, overrides=ov, loss_normalizer=N)
    print(f"  ReLU band {nb}, taken the other way {nf}", flush=True)
    assert_close("X[emb] (sampled)", v["X"][sel, 1:], c["X"][:, 1:], 2e-2)
    for name, got, ref in [("X", v["X"][sel], c["X"]), ("t", v["t"][sel, :cfg.top_in], c["t"]),
                           ("logits", v["logits"][sel], c["logits"]),
                           ("d_logits", v["d_logits"][sel], c["dz"]),
                           ("d_t", v["d_t"][sel, :cfg.top_in], g["d_top_in"]),
                           ("dX_emb", v["dX"][sel, 1:], g["dX_emb"])]:
        assert_close_composed(name + " (sampled)", got, ref, 2e-2)
    # cold rows: every occurrence's sample is in the sub-batch, so the oracle's G is exact
    Gref = np.stack([g["grad_rows"][np.searchsorted(g["unique_rows"], pos[int(uniq[u])])] for u in cold_u])
    assert_close_composed("cold grad_rows", v["grad_rows"][torch.from_numpy(cold_u).to(DEV)], Gref, 2e-2)
    assert_close_composed("cold updated rows", _rows(big["E"], uniq[cold_u]),
                          oe.sgd_rows(E_cold_before, Gref, cfg.lr_tables, round_bf16), 2e-2)
