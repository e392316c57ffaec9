"""Full-size parity of the model options at the workloads' real sizes, in
the launch configuration the benchmark times them: FP8 top layers (Section
3.5.2; the top MLP's hidden layers, or the stacked interaction's FM
projection), SwishRN with BlockNorm (Sections 3.3.4, 3.5.3), per-objective
towers (Section 3.3.3), untied top layers (Section 3.3.4) and full fusion
blocks (Section 3.3.2).  One step each (with the workload's SGD step); every
stage is recomputed by the oracle from the accelerator's own stored inputs
of that stage (the deep stack: on sampled samples, and sampled output rows
of its largest weight gradient), the interaction stages on sampled samples,
and the sparse gradient's bookkeeping in full (bit-exact) with sampled row
gradients and updates."""
import numpy as np
import pytest
import torch

import synth
from oracle import embbag as oe
from tests._util import DEV, Workload, check_sparse_stage, check_stages, grads_of

LARGE, MD, DEEP = synth.LARGE_FM, synth.MULTIDOMAIN, synth.DEEP_STACK
T = LARGE.top[-1]
OPTIONS = {
    # name: (config, fp8_top)
    "large-emb-fm-fp8-fast": (LARGE, "fast"),
    "large-emb-fm-swishrn": (LARGE.scaled(top_act="swishrn"), None),
    "large-emb-fm-towers-32": (LARGE.scaled(top=tuple(LARGE.top[:-2]) + (T * 32, T), towers=32), None),
    "multidomain-dot-untied-2": (MD.scaled(untie=2), None),
    "deep-stack-dwfb-16": (DEEP.scaled(lcb_n=16), None),
    "deep-stack-fp8-projection-fast": (DEEP.scaled(stack_fp8="fast"), None),
}


def _rows(E, rows):
    return E[torch.from_numpy(np.asarray(rows, np.int64)).to(DEV)].float().cpu().double().numpy()


@pytest.mark.gpu
@pytest.mark.parametrize("name", list(OPTIONS))
def test_fullsize_step_option(name):
    from paper_2512_09200_amd import api
    cfg, fp8 = OPTIONS[name]
    lr = cfg.lr_tables
    print(f"[fullsize-option] {name}: generating inputs", flush=True)
    w = Workload(cfg)
    b = w.batch
    bk = oe.bookkeeping(b["row_base"], b["offsets"], b["indices"], cfg.F, cfg.B)
    r = np.random.default_rng(3)
    uniq, counts = bk["unique_rows"], bk["counts"]
    sample_u = np.unique(np.concatenate([r.choice(uniq.size, 2000, replace=False),
                                         np.argsort(counts)[-10:], [0, uniq.size - 1]]))
    E_before = _rows(w.E, uniq[sample_u])
    model = w.step_model()
    lay = api.lattice_step_plan(model, cfg.B, w.nnz, lr, True, fp8_top=fp8)
    ws = torch.zeros(lay.total_bytes, dtype=torch.uint8, device=DEV)
    print(f"[fullsize-option] step (workspace {lay.total_bytes / 2**30:.2f} GiB)", flush=True)
    api.lattice_step(model, w.offsets, w.indices, w.dense, w.labels, w.mask, ws, lr, True,
                     side=api.SideStream(), fp8_top=fp8, domain_offsets=w.domain_offsets)
    torch.cuda.synchronize()
    v = api.step_views(model, ws, lay, cfg.B, cfg.T, w.nnz)
    print("[fullsize-option] stages on the accelerator's own inputs", flush=True)
    big = cfg.B > 8192
    rows = r.choice(cfg.B, 64, replace=False) if big else None
    wrows = {("top", 0): r.choice(cfg.top[0], 64, replace=False)} if big else None
    check_stages(cfg, w.params, b, v, grads_of(w), rows=rows, wgrad_rows=wrows, fp8_top=fp8)
    print("[fullsize-option] sparse gradient", flush=True)
    check_sparse_stage(cfg, b, v, w.nnz, E_before, _rows(w.E, uniq[sample_u]), lr, sample=sample_u, bk=bk)
    del w, ws
    torch.cuda.empty_cache()
