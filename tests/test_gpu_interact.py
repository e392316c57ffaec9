"""Parity of the DOT and FM interaction kernels (forward and backward)
against the oracle."""
import numpy as np
import pytest
import torch

import synth
from oracle import interact as oi
from oracle.step import rounding
from tests._util import DEV, assert_close, to_dev

CASES = {
    # name: (kind, dtype, B, n, d, k, emit0, zero_slots)
    "dot-f32-tiny": ("dot", "f32", 128, 9, 32, 0, True, False),
    "dot-bf16-n27": ("dot", "bf16", 300, 27, 64, 0, True, False),
    "dot-bf16-n97-absent": ("dot", "bf16", 96, 97, 128, 0, True, True),
    # MFMA path (bf16, n <= 128, d in {64, 128}): tile edges, no pairs, many samples per block
    "dot-bf16-n1": ("dot", "bf16", 40, 1, 64, 0, True, False),
    "dot-bf16-n2-d128": ("dot", "bf16", 40, 2, 128, 0, False, False),
    "dot-bf16-n32-d64": ("dot", "bf16", 70, 32, 64, 0, True, False),
    "dot-bf16-n33-d128": ("dot", "bf16", 70, 33, 128, 0, False, False),
    "dot-bf16-n64-d128": ("dot", "bf16", 50, 64, 128, 0, True, False),
    "dot-bf16-n128-d64-many": ("dot", "bf16", 1100, 128, 64, 0, True, False),
    "fm-bf16-n65": ("fm", "bf16", 200, 65, 128, 32, True, False),      # MFMA path
    "fm-bf16-n65-many": ("fm", "bf16", 700, 65, 128, 32, True, False), # > 1 sample per block
    "fm-bf16-n30-d64-k32": ("fm", "bf16", 37, 30, 64, 32, False, False),  # MFMA, other tiles
    "fm-bf16-n29-d128-k64": ("fm", "bf16", 41, 29, 128, 64, True, False),
    # head row (n = 32 t + 1): row 0 outside the tiles
    "fm-bf16-n33-d64-k32-head": ("fm", "bf16", 45, 33, 64, 32, False, False),
    "fm-bf16-n97-d128-k32-head": ("fm", "bf16", 600, 97, 128, 32, True, False),
    "fm-bf16-n65-d128-k64-head": ("fm", "bf16", 50, 65, 128, 64, True, False),
    "fm-bf16-n64-d128-k32": ("fm", "bf16", 60, 64, 128, 32, True, False),
    # d = 128 register-chained backward: an odd batch (last iteration one
    # sample), head and no head, rank 32 and 64, slot-0 gradient or none
    "fm-bf16-n33-d128-k32-head-odd": ("fm", "bf16", 37, 33, 128, 32, True, False),
    "fm-bf16-n64-d128-k64": ("fm", "bf16", 45, 64, 128, 64, False, False),
    "fm-bf16-n40-d128-k32": ("fm", "bf16", 515, 40, 128, 32, False, False),
    "fm-bf16-valu": ("fm", "bf16", 33, 10, 32, 16, False, False),       # VALU path (d=32)
    "fm-f32-small": ("fm", "f32", 50, 10, 32, 16, False, False),
}


@pytest.mark.gpu
@pytest.mark.parametrize("name", list(CASES))
def test_interact_fwd_bwd(name):
    print(f"[interact] {name}", flush=True)
    check_interact(*CASES[name])


@pytest.mark.gpu
@pytest.mark.parametrize("pad", [1, 3])
def test_dot_unaligned_row_stride(pad):
    """Output / gradient rows whose stride is not a multiple of 8 elements
    (the packed pairs then start off 16-byte alignment)."""
    print(f"[interact] dot n=97 d=128, row stride padded by {pad}", flush=True)
    check_interact("dot", "bf16", 33, 97, 128, 0, True, False, pad=pad)


LISTED_CASES = {
    # name: (B, n, d, emit0, fraction of zero slots, fraction of zero slots still listed, pad)
    "n97-d128-multidomain": (600, 97, 128, True, 0.58, 0.0, 0),   # > 1 sample per block
    "n97-d128-few-absent": (70, 97, 128, True, 0.1, 0.0, 0),      # 3 or 4 compact tiles
    "n27-d64": (130, 27, 64, False, 0.4, 0.0, 0),
    "n128-d64-all-listed": (40, 128, 64, True, 0.0, 0.0, 0),
    "n97-d128-zero-rows-listed": (50, 97, 128, True, 0.5, 0.5, 0),  # mask wider than the zeros
    "n97-d128-nothing-listed": (33, 97, 128, True, 1.0, 0.0, 0),   # every slot zero, mask empty
    "n97-d128-stride-pad": (45, 97, 128, True, 0.58, 0.0, 3),
    "n33-d128": (65, 33, 128, False, 0.3, 0.0, 0),
}


def _slot_mask(X, listed_zero, seed=6):
    """int32 [B, 4] bitmask: bit s set where slot s is non-zero, and for a
    fraction of the zero slots as well."""
    B, n = X.shape[:2]
    on = np.any(X != 0, axis=2)
    on |= np.random.default_rng(seed).random((B, n)) < listed_zero
    words = np.zeros((B, 4), np.uint64)
    for s_ in range(n):
        words[:, s_ // 32] |= on[:, s_].astype(np.uint64) << np.uint64(s_ % 32)
    return torch.from_numpy(words.astype(np.uint32).view(np.int32).copy()).to(DEV)


@pytest.mark.gpu
@pytest.mark.parametrize("name", list(LISTED_CASES))
def test_dot_listed_slots(name):
    """DOT with a per-sample slot mask (the kernels skip the unlisted, zero
    slots): equal to the oracle's full computation, pairs and every dX row."""
    B, n, d, emit0, zf, lz, pad = LISTED_CASES[name]
    print(f"[interact] dot listed {name}", flush=True)
    check_interact("dot", "bf16", B, n, d, 0, emit0, zf, pad=pad, listed_zero=lz)


def check_interact(kind, dt, B, n, d, k, emit0, zero_slots, pad=0, listed_zero=None):
    """Forward and backward of one interaction against the oracle; output
    rows of stride `stride + pad` (a column slice of a wider buffer).
    zero_slots: True (58%) or the fraction of slots zeroed; listed_zero not
    None: DOT with a slot mask listing the non-zero slots and that fraction
    of the zero ones."""
    from paper_2512_09200_amd import api
    rnd = rounding(dt)
    sdt = synth.torch_dtype(dt)
    t = 1e-5 if dt == "f32" else 2e-2
    X = synth.randn((B, n, d), seed=21, scale=0.05, dtype=dt)
    if zero_slots:
        r = np.random.default_rng(5)
        X[r.random((B, n)) < (0.58 if zero_slots is True else zero_slots)] = 0.0
    Xd = to_dev(X, sdt)
    mask = _slot_mask(X, listed_zero) if listed_zero is not None else None
    W = synth.randn((n, k), seed=22, scale=1 / np.sqrt(n), dtype=dt) if kind == "fm" else None
    Wd = to_dev(W, sdt) if W is not None else None
    width = (n * (n - 1) // 2 if kind == "dot" else n * k)
    off = d if emit0 else 0
    stride = (off + width + 7) // 8 * 8
    out = torch.full((B, stride + pad), 7.0, dtype=sdt, device=DEV)[:, :stride]
    api.lattice_interact_fwd(kind, Xd, out, emit_slot0=emit0, fm_W=Wd, slot_mask=mask)
    torch.cuda.synchronize()
    if kind == "dot":
        ref = oi.dot_forward(X, rnd)
    else:
        O, P = oi.fm_forward(X, W, rnd)
        ref = O.reshape(B, -1)
    assert_close("out", out[:, off:off + width], ref, t)
    if emit0:
        assert torch.equal(out[:, :d], Xd[:, 0]), "slot 0 copy"
    assert (out[:, off + width:].float() == 7.0).all(), "padding columns touched"
    # backward
    G = synth.randn((B, stride), seed=23, scale=1e-3, dtype=dt)
    Gd = torch.zeros((B, stride + pad), dtype=sdt, device=DEV)[:, :stride]
    Gd.copy_(to_dev(G, sdt))
    dX = torch.zeros((B, n, d), dtype=sdt, device=DEV)
    dW = torch.zeros((n, k), device=DEV) if kind == "fm" else None
    api.lattice_interact_bwd(kind, Xd, Gd, dX, emit_slot0=emit0, fm_W=Wd, fm_dW=dW, slot_mask=mask)
    torch.cuda.synchronize()
    if kind == "dot":
        dref = oi.dot_backward(G[:, off:off + width], X)
    else:
        dref, dWref = oi.fm_backward(G[:, off:off + width].reshape(B, n, k), X, W, P, rnd)
        assert_close("fm_dW", dW, dWref, t)
    if emit0:
        dref[:, 0] += G[:, :d]
    assert_close("dX", dX, rnd(dref), t)


STACK_CASES = {
    # name: (B, n0, stack_n, d, rank, layers, lcb_n)
    "stack-C-d64": (96, 24, 8, 64, 16, 3, 0),     # compression residual on layer 1
    "stack-id-d128": (40, 16, 16, 128, 32, 2, 0),  # identity residual throughout
    # full fusion blocks: FM block and linear compression block concatenated
    "dwfb-C-d64": (96, 24, 8, 64, 16, 3, 3),
    "dwfb-id-d128": (40, 16, 16, 128, 32, 2, 6),
    "dwfb-C-d128-lcb1": (33, 30, 10, 128, 16, 2, 1),
}


@pytest.mark.gpu
@pytest.mark.parametrize("name", list(STACK_CASES))
def test_stack_fwd_bwd(name):
    from paper_2512_09200_amd import api
    from oracle import bounds as obounds
    from tests._util import assert_close_derived, stack_dev
    B, n0, nv, d, k, L, nL = STACK_CASES[name]
    print(f"[stack] {name}", flush=True)
    cfg = synth.DEEP_STACK.scaled(B=B, F=n0, d=d, stack_n=nv, fm_rank=k, stack_layers=L,
                                  lcb_n=nL, top=(16, 4), seed=77)
    params = synth.make_dense_params(cfg)
    layers = params["stack"]
    rnd = rounding("bf16")
    X = synth.randn((B, n0, d), seed=31, scale=0.05, dtype="bf16")
    Xd = to_dev(X, torch.bfloat16)
    dev_layers = stack_dev(layers, torch.bfloat16)
    out = torch.zeros((B, nv * d), dtype=torch.bfloat16, device=DEV)
    ws = api.lattice_interact_fwd("stack", Xd, out, stack=dev_layers, stack_n=nv, ln_eps=cfg.ln_eps)
    torch.cuda.synchronize()
    XL, caches = oi.stack_forward(X, layers, nv, d, rnd, cfg.ln_eps)
    G = synth.randn((B, nv * d), seed=32, scale=1e-3, dtype="bf16")
    dX = torch.zeros((B, n0, d), dtype=torch.bfloat16, device=DEV)
    api.lattice_interact_bwd("stack", Xd, to_dev(G, torch.bfloat16), dX, stack=dev_layers,
                             stack_n=nv, ln_eps=cfg.ln_eps, ws=ws)
    torch.cuda.synchronize()
    dY = np.asarray(G, np.float64).reshape(B, nv, d)
    dX1, grads = oi.stack_backward(dY, layers, caches, rnd)
    zero = lambda x: (np.zeros(x.shape), np.zeros(x.shape))
    Xf = np.asarray(X, np.float64)
    e_out, edX, eg = obounds.stack_bounds(Xf, zero(Xf), dY, zero(dY), layers, caches, "bf16")
    # three layers deep: element-wise within the tolerance or the deviation
    # the arithmetic itself allows (oracle.bounds)
    assert_close_derived("X_L", out, XL.reshape(B, -1), (e_out[0].reshape(B, -1), e_out[1].reshape(B, -1)),
                         2e-2)
    assert_close_derived("dX", dX, rnd(dX1), obounds.rounded(edX, dX1, 2.0 ** -8), 2e-2)
    for l, (gl, dl, el) in enumerate(zip(grads, dev_layers, eg)):
        for key in ("dW", "dA", "dgamma", "dC", "dL"):
            if key in gl:
                assert_close_derived(f"layer{l}.{key}", dl[key], gl[key], el[key], 2e-2)


FP8_STACK_CASES = {
    # name: (B, n0, stack_n, d, rank, layers, lcb_n, fp8 accumulation)
    "stack-C-d64-fp8-precise": (96, 24, 8, 64, 16, 3, 0, "precise"),
    "stack-id-d128-fp8-fast": (40, 16, 16, 128, 32, 2, 0, "fast"),
    "dwfb-C-d128-fp8-precise": (33, 30, 10, 128, 16, 2, 1, "precise"),
    "stack-C-d128-fp8-fast-long-rows": (20, 64, 32, 128, 64, 2, 0, "fast"),   # vec(F) rows of 4096
}


@pytest.mark.gpu
@pytest.mark.parametrize("name", list(FP8_STACK_CASES))
def test_stack_fp8_projection(name):
    """The stacked interaction with its FM projection vec(F) A^T in FP8
    (Section 3.5.2), stage by stage from the GPU's own saved state
    (tests._util.check_stack_fp8): the FP8 product within the accumulation
    bound of the exact product of the codes, LayerNorm from the stored H,
    and the bf16 backward (the quantisation taken as the identity) through
    the oracle from the GPU's forward values."""
    from paper_2512_09200_amd import api
    from oracle import bounds as obounds
    from tests._util import assert_close_derived, check_stack_fp8, stack_dev
    B, n0, nv, d, k, L, nL, mode = FP8_STACK_CASES[name]
    print(f"[stack-fp8] {name}", flush=True)
    cfg = synth.DEEP_STACK.scaled(B=B, F=n0, d=d, stack_n=nv, fm_rank=k, stack_layers=L,
                                  lcb_n=nL, top=(16, 4), seed=78)
    params = synth.make_dense_params(cfg)
    layers = params["stack"]
    rnd = rounding("bf16")
    X = synth.randn((B, n0, d), seed=33, scale=0.05, dtype="bf16")
    Xd = to_dev(X, torch.bfloat16)
    dev_layers = stack_dev(layers, torch.bfloat16)
    out = torch.zeros((B, nv * d), dtype=torch.bfloat16, device=DEV)
    ws = api.lattice_interact_fwd("stack", Xd, out, stack=dev_layers, stack_n=nv, ln_eps=cfg.ln_eps,
                                  fp8_proj=mode)
    G = synth.randn((B, nv * d), seed=34, scale=1e-3, dtype="bf16")
    dX = torch.zeros((B, n0, d), dtype=torch.bfloat16, device=DEV)
    api.lattice_interact_bwd("stack", Xd, to_dev(G, torch.bfloat16), dX, stack=dev_layers,
                             stack_n=nv, ln_eps=cfg.ln_eps, ws=ws, fp8_proj=mode)
    torch.cuda.synchronize()
    state = api.lattice_interact_state("stack", Xd, dev_layers, nv, ws, ln_eps=cfg.ln_eps, fp8_proj=mode)
    dX1, grads, edX, eg = check_stack_fp8(layers, X, state, out, G, None, None, mode, cfg.ln_eps)
    assert_close_derived("dX", dX, rnd(dX1), obounds.rounded(edX, dX1, 2.0 ** -8), 2e-2)
    for l, (gl, dl, el) in enumerate(zip(grads, dev_layers, eg)):
        for key in ("dW", "dA", "dgamma", "dC", "dL"):
            if key in gl:
                assert_close_derived(f"layer{l}.{key}", dl[key], gl[key], el[key], 2e-2)
