"""The step's forward alone (lattice_forward, the inference path; Section
3.5.2 serves with FP8 and fast accumulation): the same kernels in the same
order as the forward of lattice_step, so its logits and forward
intermediates equal the step's bit for bit (the step's forward is held to
the oracle in test_gpu_step.py); labels are not read.  One configuration is
also compared with the oracle's forward directly."""
import pytest
import torch

import synth
from oracle import step as ostep
from oracle import bounds as obounds
from tests._util import DEV, Workload, assert_close_derived, relu_overrides

CASES = {
    # name: (config, fp8_top)
    "large-fm-small": (synth.small(synth.LARGE_FM, B=128, rows=6000), None),
    "large-fm-small-fp8-fast": (synth.small(synth.LARGE_FM, B=128, rows=6000), "fast"),
    "mid-small": (synth.small(synth.MID, B=256, rows=3000), None),
    "multidomain-small": (synth.small(synth.MULTIDOMAIN, B=256, rows=2000), None),
    "multidomain-small-untied": (synth.small(synth.MULTIDOMAIN, B=256, rows=2000, untie=2), None),
    "mid-small-swishrn-towers": (synth.small(synth.MID, B=200, rows=3000, top=(512, 8 * 32, 8), towers=32,
                                             top_act="swishrn"), None),
    "tiny-f32": (synth.TINY, None),
    "deep-stack-small": (synth.DEEP_STACK.scaled(B=48, F=32, rows=1000, stack_n=16, fm_rank=32,
                                                 top=(256, 64, 16), lcb_n=4), None),
}


def _run(w, fp8, forward_only):
    from paper_2512_09200_amd import api
    cfg = w.cfg
    model = w.step_model()
    lay = api.lattice_step_plan(model, cfg.B, w.nnz, 0.0, True, fp8_top=fp8)
    ws = torch.zeros(lay.total_bytes, dtype=torch.uint8, device=DEV)
    if forward_only:
        api.lattice_forward(model, w.offsets, w.indices, w.dense, cfg.B, ws, side=api.SideStream(),
                            fp8_top=fp8, domain_offsets=w.domain_offsets)
    else:
        api.lattice_step(model, w.offsets, w.indices, w.dense, w.labels, w.mask, ws, 0.0, True,
                         side=api.SideStream(), fp8_top=fp8, domain_offsets=w.domain_offsets)
    torch.cuda.synchronize()
    return api.step_views(model, ws, lay, cfg.B, cfg.T, w.nnz)


@pytest.mark.gpu
@pytest.mark.parametrize("name", list(CASES))
def test_forward_alone_equals_the_steps_forward(name):
    cfg, fp8 = CASES[name]
    print(f"[forward] {name} B={cfg.B} fp8={fp8}", flush=True)
    w = Workload(cfg)
    v_step = _run(w, fp8, False)
    v_fwd = _run(w, fp8, True)
    assert torch.equal(v_fwd["logits"], v_step["logits"]), "logits"
    assert torch.equal(v_fwd["X"], v_step["X"]), "stacked vectors"
    assert torch.equal(v_fwd["t"], v_step["t"]), "top input"
    for i, (a, b) in enumerate(zip(v_fwd["top_act"], v_step["top_act"])):
        assert torch.equal(a, b), f"top activation {i}"
    assert torch.isfinite(v_fwd["logits"]).all()


@pytest.mark.gpu
def test_forward_alone_matches_oracle():
    """large-fm-small: the logits of the forward alone against the oracle's
    forward from the same inputs, element-wise or within the derived
    deviation of the composed forward (bf16 storage points)."""
    from tests.test_gpu_step import gpu_relu_io
    cfg = synth.small(synth.LARGE_FM, B=128, rows=6000)
    w = Workload(cfg)
    E0 = w.table_np()
    v = _run(w, None, True)
    # ReLU decisions inside the fp32 ambiguity band taken as the GPU took them
    ov, nband, nflip = relu_overrides(cfg, w.params, E0, w.batch, *gpu_relu_io(cfg, w, v))
    print(f"  ReLU decisions in the band: {nband}, taken the other way: {nflip}", flush=True)
    c, g = ostep.step(cfg, w.params, E0, w.batch, lr_tables=0.0, overrides=ov)
    bd = obounds.step_bounds(cfg, w.params, E0, w.batch, c, g, lr_tables=0.0)
    assert_close_derived("t (forward alone)", v["t"][:, :cfg.top_in], c["t"], bd["t"], 2e-2)
    assert_close_derived("logits (forward alone)", v["logits"], c["logits"], bd["logits"], 2e-2)
