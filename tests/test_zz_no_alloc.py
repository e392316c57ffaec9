"""The allocation-free sparse gradient (lattice_embbag_bwd_noalloc) against
the workspace entry point (lattice_embbag_bwd) through the C ABI: two calls
in a row on one GPU, the second with a smaller batch (the shared scratch
keeps the first call's contents), each bit-identical to the workspace
entry point on the same inputs (the same kernels in the same order:
bookkeeping, row gradients and SGD-updated tables), and a batch beyond the
scratch's capacity rejected before anything is launched."""
import numpy as np
import pytest
import torch

import synth
from tests._util import DEV

CASES = [synth.small(synth.LARGE_FM, B=512, rows=20000), synth.small(synth.MID, B=96, rows=3000)]


def _inputs(cfg):
    b = synth.make_batch(cfg)
    E = synth.make_tables(cfg, device=DEV)
    dX = torch.from_numpy(synth.randn((cfg.B, cfg.n_slots, cfg.d), seed=cfg.seed, stream=9, scale=1e-2,
                                      dtype=cfg.dtype)).to(synth.torch_dtype(cfg.dtype)).to(DEV)
    return (E, torch.from_numpy(b["row_base"]).to(DEV), torch.from_numpy(b["offsets"]).to(DEV),
            torch.from_numpy(b["indices"]).to(DEV), dX, int(b["offsets"][-1]))


def _outputs(nnz, d):
    n = max(nnz, 1)
    return dict(unique_rows=torch.full((n,), -7, dtype=torch.int32, device=DEV),
                seg_offsets=torch.full((n + 1,), -7, dtype=torch.int32, device=DEV),
                sorted_bags=torch.full((n,), -7, dtype=torch.int32, device=DEV),
                num_unique=torch.full((1,), -7, dtype=torch.int32, device=DEV),
                grad_rows=torch.full((n, d), float("nan"), device=DEV))


@pytest.mark.gpu
def test_noalloc_matches_workspace_entry_point_on_consecutive_calls():
    from paper_2512_09200_amd import api
    for k, cfg in enumerate(CASES):           # the second call has fewer lookups
        E, row_base, offsets, indices, dX, nnz = _inputs(cfg)
        print(f"[noalloc] call {k}: {cfg.name} B={cfg.B} nnz={nnz}", flush=True)
        lr = 0.5
        E_ws, E_na = E.clone(), E.clone()
        ref = api.lattice_embbag_bwd(E_ws, row_base, offsets, indices, cfg.F, cfg.B, dX, first_slot=1, lr=lr)
        out = api.lattice_embbag_bwd_noalloc(E_na, row_base, offsets, indices, cfg.F, cfg.B, dX,
                                             _outputs(nnz, cfg.d), first_slot=1, lr=lr)
        torch.cuda.synchronize()
        U = int(ref["num_unique"].item())
        assert U > 0 and int(out["num_unique"].item()) == U
        for key, n in (("unique_rows", U), ("seg_offsets", U + 1), ("sorted_bags", nnz), ("grad_rows", U)):
            assert torch.equal(out[key][:n], ref[key][:n]), key
        assert torch.equal(E_na, E_ws)
        assert not torch.equal(E_na, E)          # the SGD step did move rows
        del E, E_ws, E_na
        torch.cuda.empty_cache()


@pytest.mark.gpu
def test_noalloc_rejects_batches_beyond_its_scratch():
    from paper_2512_09200_amd import api
    from paper_2512_09200_amd._abi import LatticeError
    nnz = 17_000_000                          # needs ~270 MiB of scratch at dim 128
    E = torch.zeros((1000, 128), dtype=torch.bfloat16, device=DEV)
    row_base = torch.tensor([0, 1000], dtype=torch.int64, device=DEV)
    offsets = torch.tensor([0, nnz], dtype=torch.int32, device=DEV)
    indices = torch.zeros(nnz, dtype=torch.int32, device=DEV)
    dX = torch.zeros((1, 2, 128), dtype=torch.bfloat16, device=DEV)
    out = _outputs(1, 128)
    with pytest.raises(LatticeError, match="UNSUPPORTED"):
        api.lattice_embbag_bwd_noalloc(E, row_base, offsets, indices, 1, 1, dX, out, first_slot=1)
    torch.cuda.synchronize()
    assert int(out["num_unique"].item()) == -7   # nothing was launched
