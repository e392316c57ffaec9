"""Parity of the pooled lookup and its deterministic sparse gradient against
the oracle (bookkeeping bit-exact; values to the workload's tolerance)."""
import numpy as np
import pytest
import torch

import synth
from oracle import embbag as oe
from oracle.step import rounding
from tests._util import DEV, Workload, assert_close, tol

CASES = {
    "tiny": synth.TINY,
    "tiny-mean": synth.TINY.scaled(pool="mean"),
    "mid-small": synth.small(synth.MID, B=256, rows=3000),
    "multidomain-small-empty-bags": synth.small(synth.MULTIDOMAIN, B=192, rows=1500),
    "large-fm-small": synth.small(synth.LARGE_FM, B=64, rows=20000),
    "d256-bf16-mean": synth.small(synth.MID, B=96, rows=800, F=5, d=256, pool="mean"),
    # ~20K lookups per feature: several sort tiles per segment and a ragged last one
    "mid-multitile": synth.small(synth.MID, B=2048, rows=100000, F=3),
}


def _X(w, fill):
    c = w.cfg
    return torch.full((c.B, c.n_slots, c.d), fill, dtype=synth.torch_dtype(c.dtype), device=DEV)


@pytest.mark.gpu
@pytest.mark.parametrize("name", list(CASES))
def test_embbag_fwd(name):
    from paper_2512_09200_amd import api
    cfg = CASES[name]
    print(f"[embbag_fwd] {name} B={cfg.B} F={cfg.F} d={cfg.d} {cfg.dtype}", flush=True)
    w = Workload(cfg)
    X = _X(w, float("nan"))
    api.lattice_embbag_fwd(w.E, w.row_base, w.offsets, w.indices, cfg.F, cfg.B, X,
                           cfg.first_emb_slot, cfg.pool)
    torch.cuda.synchronize()
    ref = rounding(cfg.dtype)(oe.pool_forward(w.table_np(), w.batch["row_base"], w.batch["offsets"],
                                              w.batch["indices"], cfg.F, cfg.B, cfg.pool))
    assert_close("X", X[:, cfg.first_emb_slot:], ref, tol(cfg))
    if cfg.first_emb_slot:
        assert torch.isnan(X[:, 0].float()).all(), "slot 0 must not be touched"
    empty = np.diff(w.batch["offsets"]).reshape(cfg.F, cfg.B) == 0
    if empty.any():
        got = X[:, cfg.first_emb_slot:].float().cpu().numpy().transpose(1, 0, 2)
        assert np.all(got[empty] == 0), "empty bags must pool to exact zeros"


@pytest.mark.gpu
@pytest.mark.parametrize("name", list(CASES))
@pytest.mark.parametrize("lr", [0.0, 0.5])
def test_embbag_bwd(name, lr):
    from paper_2512_09200_amd import api
    cfg = CASES[name]
    print(f"[embbag_bwd] {name} lr={lr}", flush=True)
    w = Workload(cfg)
    rnd = rounding(cfg.dtype)
    dX_np = synth.randn((cfg.B, cfg.n_slots, cfg.d), seed=cfg.seed, stream=1, scale=1e-2,
                        dtype=cfg.dtype)
    dX = torch.from_numpy(dX_np).to(synth.torch_dtype(cfg.dtype)).to(DEV)
    E0 = w.table_np()
    out = api.lattice_embbag_bwd(w.E, w.row_base, w.offsets, w.indices, cfg.F, cfg.B, dX,
                                 cfg.first_emb_slot, lr=lr, pool=cfg.pool)
    torch.cuda.synchronize()
    b = w.batch
    bk = oe.bookkeeping(b["row_base"], b["offsets"], b["indices"], cfg.F, cfg.B)
    uniq, G = oe.pool_backward(dX_np[:, cfg.first_emb_slot:], b["row_base"], b["offsets"],
                               b["indices"], cfg.F, cfg.B, cfg.pool)
    U = int(out["num_unique"].item())
    assert U == uniq.size
    np.testing.assert_array_equal(out["unique_rows"][:U].cpu().numpy(), bk["unique_rows"])
    seg = np.append(bk["seg_offsets"], w.nnz)
    np.testing.assert_array_equal(out["seg_offsets"][:U + 1].cpu().numpy(), seg)
    np.testing.assert_array_equal(out["sorted_bags"][:w.nnz].cpu().numpy(), bk["sorted_bags"])
    assert_close("grad_rows", out["grad_rows"][:U], G, tol(cfg))
    E1 = w.table_np()
    if lr:
        assert_close("updated_rows", E1[uniq], oe.sgd_rows(E0[uniq], G, lr, rnd), tol(cfg))
        untouched = np.ones(E0.shape[0], bool)
        untouched[uniq] = False
        assert np.array_equal(E1[untouched], E0[untouched]), "untouched rows changed"
    else:
        assert np.array_equal(E1, E0)


@pytest.mark.gpu
def test_embbag_bwd_hot_row_spanning_many_chunks():
    """One row hit 5000 times in a bag plus singles: a run spanning ~80 chunks."""
    from paper_2512_09200_amd import api
    cfg = synth.Config(name="hot", B=4, F=2, rows=1000, d=64, dtype="bf16", index_dist=("uniform",),
                       bag_dist=("uniform", 1, 1), dense_in=0, bottom=(), interact="dot", top=(1,))
    lens = np.array([5000, 1, 3, 0, 7, 2, 0, 1])
    offsets = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    idx = np.concatenate([np.full(5000, 17), [3], [17, 17, 999], [5, 6, 17, 17, 0, 999, 998], [1, 1], [17]]).astype(np.int32)
    row_base = np.array([0, 1000, 2000])
    E = torch.randn((2000, 64), device=DEV).mul_(0.01).to(torch.bfloat16)
    dX_np = synth.randn((4, 2, 64), seed=5, stream=2, dtype="bf16")
    dX = torch.from_numpy(dX_np).to(torch.bfloat16).to(DEV)
    E0 = E.float().cpu().double().numpy()
    out = api.lattice_embbag_bwd(E, torch.from_numpy(row_base).to(DEV), torch.from_numpy(offsets).to(DEV),
                                 torch.from_numpy(idx).to(DEV), 2, 4, dX, 0, lr=0.25)
    torch.cuda.synchronize()
    bk = oe.bookkeeping(row_base, offsets, idx, 2, 4)
    uniq, G = oe.pool_backward(dX_np, row_base, offsets, idx, 2, 4)
    U = int(out["num_unique"].item())
    np.testing.assert_array_equal(out["unique_rows"][:U].cpu().numpy(), bk["unique_rows"])
    np.testing.assert_array_equal(out["sorted_bags"][:idx.size].cpu().numpy(), bk["sorted_bags"])
    assert_close("grad_rows", out["grad_rows"][:U], G, 2e-2)
    E1 = E.float().cpu().double().numpy()
    from oracle.bf16 import round_bf16
    assert_close("updated_rows", E1[uniq], oe.sgd_rows(E0[uniq], G, 0.25, round_bf16), 2e-2)


@pytest.mark.gpu
def test_embbag_bwd_is_deterministic():
    from paper_2512_09200_amd import api
    cfg = CASES["mid-small"]
    w = Workload(cfg)
    dX = torch.from_numpy(synth.randn((cfg.B, cfg.n_slots, cfg.d), seed=9, dtype=cfg.dtype)).to(
        torch.bfloat16).to(DEV)
    r1 = api.lattice_embbag_bwd(w.E, w.row_base, w.offsets, w.indices, cfg.F, cfg.B, dX, 1)
    r2 = api.lattice_embbag_bwd(w.E, w.row_base, w.offsets, w.indices, cfg.F, cfg.B, dX, 1)
    torch.cuda.synchronize()
    U = int(r1["num_unique"].item())
    assert U == int(r2["num_unique"].item())
    # only the first num_unique entries (num_unique+1 offsets) are defined
    for k, n in (("unique_rows", U), ("seg_offsets", U + 1), ("sorted_bags", w.nnz), ("grad_rows", U)):
        assert torch.equal(r1[k][:n], r2[k][:n]), k


@pytest.mark.gpu
def test_validate_batch():
    from paper_2512_09200_amd import api
    cfg = CASES["mid-small"]
    w = Workload(cfg)
    ok, _ = api.lattice_validate_batch(w.E, w.row_base, w.offsets, w.indices, cfg.F, cfg.B)
    assert ok
    bad = w.indices.clone()
    bad[123] = cfg.rows          # one past the end of its table
    ok, pos = api.lattice_validate_batch(w.E, w.row_base, w.offsets, bad, cfg.F, cfg.B)
    assert not ok and pos == 123
    off = w.offsets.clone()
    off[10] = off[11] + 1        # non-monotone
    ok, pos = api.lattice_validate_batch(w.E, w.row_base, off, w.indices, cfg.F, cfg.B)
    assert not ok and pos < 0
    # a row bound smaller than the tables
    ok, pos = api.lattice_validate_batch(w.E, w.row_base, w.offsets, w.indices, cfg.F, cfg.B,
                                         max_rows=cfg.rows - 1)
    assert not ok and pos == -1 - (cfg.F * cfg.B + 1)


@pytest.mark.gpu
def test_embbag_bwd_row_bound_only_changes_passes():
    """The backward sorts each feature by its local row with as many digit
    passes as max_rows needs; with max_rows unknown (0) it uses the total row
    count (more passes).  Both must give identical results."""
    from paper_2512_09200_amd import api
    cfg = CASES["large-fm-small"]
    w = Workload(cfg)
    dX = torch.from_numpy(synth.randn((cfg.B, cfg.n_slots, cfg.d), seed=11, dtype=cfg.dtype)).to(
        torch.bfloat16).to(DEV)
    r1 = api.lattice_embbag_bwd(w.E, w.row_base, w.offsets, w.indices, cfg.F, cfg.B, dX, 1, max_rows=0)
    r2 = api.lattice_embbag_bwd(w.E, w.row_base, w.offsets, w.indices, cfg.F, cfg.B, dX, 1)
    torch.cuda.synchronize()
    U = int(r1["num_unique"].item())
    assert U == int(r2["num_unique"].item())
    for k, n in (("unique_rows", U), ("seg_offsets", U + 1), ("sorted_bags", w.nnz), ("grad_rows", U)):
        assert torch.equal(r1[k][:n], r2[k][:n]), k


def _structured_bags(rng, F, B, rows):
    """Bags whose sorted occurrence list has runs of lengths around the
    256-occurrence reduction ranges: runs of exactly 256 and 257, a run of
    255 + 1, a run of 1000, then a mix of singles and short runs."""
    runs = [256, 257, 255, 1, 1000, 3, 512, 1, 1, 2, 64, 65, 300]
    idx_per_feature = [[] for _ in range(F)]
    r = 0
    for L in runs:
        f = r % F
        idx_per_feature[f].extend([(17 * r + 5) % rows] * L)
        r += 1
    for f in range(F):
        idx_per_feature[f].extend(rng.integers(0, rows, size=int(rng.integers(50, 400))).tolist())
        rng.shuffle(idx_per_feature[f])
    offsets = [0]
    indices = []
    for f in range(F):
        ids = idx_per_feature[f]
        cuts = np.sort(rng.integers(0, len(ids) + 1, size=B - 1))
        cuts = np.concatenate([[0], cuts, [len(ids)]])
        for b in range(B):
            indices.extend(ids[cuts[b]:cuts[b + 1]])
            offsets.append(len(indices))
    return np.array(offsets, np.int32), np.array(indices, np.int32)


LANE_LAYOUTS = [(8, "bf16", "sum"), (16, "bf16", "mean"), (24, "bf16", "sum"), (32, "bf16", "sum"),
                (40, "f32", "sum"), (128, "bf16", "mean"), (256, "f32", "sum"), (256, "bf16", "sum")]


@pytest.mark.gpu
@pytest.mark.parametrize("d,dtype,pool", LANE_LAYOUTS, ids=[f"d{d}-{t}-{p}" for d, t, p in LANE_LAYOUTS])
@pytest.mark.parametrize("lr", [0.0, 0.25])
def test_embbag_bwd_range_boundaries(d, dtype, pool, lr):
    """Runs that end exactly at, one before and one after the 256-occurrence
    reduction ranges, plus long runs crossing several, at every lane layout of
    the reduction (16-byte lanes per row from 1 to 64, and widths that are not
    a power of two)."""
    from paper_2512_09200_amd import api
    print(f"[embbag_bwd_ranges] d={d} {dtype} {pool} lr={lr}", flush=True)
    F, B, rows = 3, 37, 700
    rng = np.random.default_rng(20251209 + d)
    offsets, idx = _structured_bags(rng, F, B, rows)
    row_base = np.arange(F + 1, dtype=np.int64) * rows
    sdt = synth.torch_dtype(dtype)
    E = torch.from_numpy(synth.randn((F * rows, d), seed=d, stream=3, scale=0.1, dtype=dtype)).to(sdt).to(DEV)
    dX_np = synth.randn((B, F + 1, d), seed=d, stream=4, dtype=dtype)
    dX = torch.from_numpy(dX_np).to(sdt).to(DEV)
    E0 = E.float().cpu().double().numpy()
    out = api.lattice_embbag_bwd(E, torch.from_numpy(row_base).to(DEV), torch.from_numpy(offsets).to(DEV),
                                 torch.from_numpy(idx).to(DEV), F, B, dX, 1, lr=lr, pool=pool)
    torch.cuda.synchronize()
    bk = oe.bookkeeping(row_base, offsets, idx, F, B)
    uniq, G = oe.pool_backward(dX_np[:, 1:], row_base, offsets, idx, F, B, pool)
    U = int(out["num_unique"].item())
    assert U == uniq.size
    np.testing.assert_array_equal(out["unique_rows"][:U].cpu().numpy(), bk["unique_rows"])
    np.testing.assert_array_equal(out["seg_offsets"][:U + 1].cpu().numpy(), np.append(bk["seg_offsets"], idx.size))
    np.testing.assert_array_equal(out["sorted_bags"][:idx.size].cpu().numpy(), bk["sorted_bags"])
    t = 1e-5 if dtype == "f32" else 2e-2
    assert_close("grad_rows", out["grad_rows"][:U], G, t)
    E1 = E.float().cpu().double().numpy()
    if lr:
        assert_close("updated_rows", E1[uniq], oe.sgd_rows(E0[uniq], G, lr, rounding(dtype)), t)
        untouched = np.ones(E0.shape[0], bool)
        untouched[uniq] = False
        assert np.array_equal(E1[untouched], E0[untouched]), "untouched rows changed"
    else:
        assert np.array_equal(E1, E0)


MIXED = [(128, "bf16", "f32"), (64, "f32", "bf16"), (32, "bf16", "f32"), (256, "f32", "bf16")]


@pytest.mark.gpu
@pytest.mark.parametrize("d,dx_dtype,table_dtype", MIXED, ids=[f"d{d}-dX{a}-E{b}" for d, a, b in MIXED])
def test_embbag_bwd_mixed_dtypes(d, dx_dtype, table_dtype):
    """The gradient's storage dtype differs from the table's: the table rows
    are addressed by their own width (dX rows of 256 bytes with 512- or
    128-byte table rows included)."""
    from paper_2512_09200_amd import api
    print(f"[embbag_bwd_mixed] d={d} dX {dx_dtype} table {table_dtype}", flush=True)
    F, B, rows, lr = 3, 37, 700, 0.25
    rng = np.random.default_rng(77 + d)
    offsets, idx = _structured_bags(rng, F, B, rows)
    row_base = np.arange(F + 1, dtype=np.int64) * rows
    E = torch.from_numpy(synth.randn((F * rows, d), seed=d, stream=5, scale=0.1, dtype=table_dtype)).to(
        synth.torch_dtype(table_dtype)).to(DEV)
    dX_np = synth.randn((B, F + 1, d), seed=d, stream=6, dtype=dx_dtype)
    dX = torch.from_numpy(dX_np).to(synth.torch_dtype(dx_dtype)).to(DEV)
    E0 = E.float().cpu().double().numpy()
    out = api.lattice_embbag_bwd(E, torch.from_numpy(row_base).to(DEV), torch.from_numpy(offsets).to(DEV),
                                 torch.from_numpy(idx).to(DEV), F, B, dX, 1, lr=lr)
    torch.cuda.synchronize()
    uniq, G = oe.pool_backward(dX_np[:, 1:], row_base, offsets, idx, F, B, "sum")
    U = int(out["num_unique"].item())
    assert U == uniq.size
    # dX values are exact in fp64: the fp32 sums are within fp32 rounding
    assert_close("grad_rows", out["grad_rows"][:U], G, 1e-5)
    E1 = E.float().cpu().double().numpy()
    t = 1e-5 if table_dtype == "f32" else 2e-2
    assert_close("updated_rows", E1[uniq], oe.sgd_rows(E0[uniq], G, lr, rounding(table_dtype)), t)
    untouched = np.ones(E0.shape[0], bool)
    untouched[uniq] = False
    assert np.array_equal(E1[untouched], E0[untouched]), "untouched rows changed"


@pytest.mark.gpu
@pytest.mark.parametrize("rows", [(1 << 24) - 1, (1 << 24) + 1], ids=["span-4GiB-minus-256B", "span-over-4GiB"])
def test_embbag_bwd_far_apart_rows(rows):
    """A 4 GiB bf16 table (d=128, 256-byte rows) whose first and last rows
    occur in the same reduction range: the rows such a range touches span
    just under 4 GiB (one buffer window) or just over it (64-bit row
    addresses).  The table is zero except the touched rows; only those and
    their neighbours are compared."""
    from paper_2512_09200_amd import api
    print(f"[embbag_bwd_far] rows={rows}", flush=True)
    d, F, B, lr = 128, 1, 8, 0.5
    touched = np.array([0, 1, 5, rows // 2, rows - 3, rows - 1], np.int64)
    rng = np.random.default_rng(rows)
    idx = rng.choice(touched, size=40).astype(np.int32)
    idx[:2] = [0, rows - 1]
    cuts = np.sort(rng.integers(0, idx.size + 1, size=B - 1))
    offsets = np.concatenate([[0], cuts, [idx.size]]).astype(np.int32)
    row_base = np.array([0, rows], np.int64)
    E = torch.zeros((rows, d), dtype=torch.bfloat16, device=DEV)
    look = np.unique(np.clip(np.concatenate([touched - 1, touched, touched + 1]), 0, rows - 1))
    vals = torch.from_numpy(synth.randn((look.size, d), seed=3, stream=7, scale=0.1, dtype="bf16")).to(
        torch.bfloat16).to(DEV)
    look_t = torch.from_numpy(look).to(DEV)
    E[look_t] = vals
    E0 = E[look_t].float().cpu().double().numpy()
    dX_np = synth.randn((B, F, d), seed=4, stream=8, dtype="bf16")
    dX = torch.from_numpy(dX_np).to(torch.bfloat16).to(DEV)
    out = api.lattice_embbag_bwd(E, torch.from_numpy(row_base).to(DEV), torch.from_numpy(offsets).to(DEV),
                                 torch.from_numpy(idx).to(DEV), F, B, dX, 0, lr=lr)
    torch.cuda.synchronize()
    uniq, G = oe.pool_backward(dX_np, row_base, offsets, idx, F, B, "sum")
    U = int(out["num_unique"].item())
    assert U == uniq.size
    np.testing.assert_array_equal(out["unique_rows"][:U].cpu().numpy(), uniq)
    assert_close("grad_rows", out["grad_rows"][:U], G, 1e-5)
    E1 = E[look_t].float().cpu().double().numpy()
    pos = np.searchsorted(look, uniq)
    assert_close("updated_rows", E1[pos], oe.sgd_rows(E0[pos], G, lr, rounding("bf16")), 2e-2)
    other = np.ones(look.size, bool)
    other[pos] = False
    assert np.array_equal(E1[other], E0[other]), "untouched rows changed"
    del E
    torch.cuda.empty_cache()
