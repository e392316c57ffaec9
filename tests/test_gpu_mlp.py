"""Parity of the MLP/heads GEMM path (forward, masked BCE, backward) against
the oracle, on shapes that span several 128x128 tiles with ragged tails, odd
K (element loader) and aligned K (vector loaders)."""
import numpy as np
import pytest
import torch

import synth
from oracle import loss as oloss
from oracle import mlp as omlp
from oracle.step import rounding
from tests._util import DEV, assert_close, to_dev

SHAPES = {
    # name: (dtype, B, dims, relu_last)
    "bf16-aligned-heads": ("bf16", 300, (64, 256, 136, 8), False),
    "bf16-odd-heads": ("bf16", 257, (77, 130, 5), False),
    "bf16-bottom": ("bf16", 200, (13, 256, 64), True),
    "f32-heads": ("f32", 128, (68, 64, 4), False),
    "f32-bottom": ("f32", 129, (13, 64, 32), True),
    "bf16-deep-k": ("bf16", 512, (2208, 1024, 16), False),
    # input rows padded to 8 elements (NaN in the padding): vector loads of
    # the last partial vector must not let the padding into the contraction
    "bf16-padded-in-415": ("bf16", 300, (415, 512, 256, 8), False),
    "bf16-padded-in-13": ("bf16", 260, (13, 256, 64), True),
    # products with >= 256 tiles of 256x256 (the large-tile kernel): forward
    # with bias + ReLU, and the second layer's input gradient with the ReLU
    # mask; ragged M, N and K edges
    "bf16-big-tiles": ("bf16", 4000, (1032, 4040, 8), False),
}
PADDED = {"bf16-padded-in-415", "bf16-padded-in-13"}


def _layers(dt, dims, seed):
    r = np.random.default_rng(seed)
    out = []
    for i in range(len(dims) - 1):
        W = synth.to_storage(r.standard_normal((dims[i + 1], dims[i])) * np.sqrt(2 / (dims[i] + dims[i + 1])), dt).float().numpy()
        b = (r.standard_normal(dims[i + 1]) * 0.01).astype(np.float32)
        out.append((W, b))
    return out


@pytest.mark.gpu
@pytest.mark.parametrize("name", list(SHAPES))
def test_mlp_fwd_bwd(name):
    from paper_2512_09200_amd import api
    dt, B, dims, relu_last = SHAPES[name]
    print(f"[mlp] {name}", flush=True)
    rnd = rounding(dt)
    sdt = synth.torch_dtype(dt)
    t = 1e-5 if dt == "f32" else 2e-2
    layers = _layers(dt, dims, 11)
    x = synth.randn((B, dims[0]), seed=12, dtype=dt)
    L = [dict(W=to_dev(W, sdt), b=to_dev(b), dW=torch.zeros(W.shape, device=DEV),
              db=torch.zeros(b.shape, device=DEV)) for W, b in layers]
    xd = to_dev(x, sdt)
    if name in PADDED:
        ld = (dims[0] + 7) // 8 * 8
        buf = torch.full((B, ld), float("nan"), dtype=sdt, device=DEV)
        buf[:, :dims[0]] = xd
        xd = buf[:, :dims[0]]
    acts = [torch.empty((B, dims[i + 1]), dtype=(torch.float32 if (i == len(layers) - 1 and not relu_last) else sdt),
                        device=DEV) for i in range(len(layers))]
    loss = None
    if not relu_last:
        T = dims[-1]
        y = (np.random.default_rng(3).random((B, T)) < 0.3).astype(np.float32)
        m = (np.random.default_rng(4).random((B, T)) < 0.5).astype(np.uint8)
        loss = dict(labels=to_dev(y), mask=to_dev(m), loss=torch.zeros(1, device=DEV),
                    d_logits=torch.zeros((B, T), device=DEV),
                    d_logits_op=torch.zeros((B, T), dtype=sdt, device=DEV))
    api.lattice_mlp_heads_fwd(L, xd, acts, relu_last, loss)
    torch.cuda.synchronize()
    # ReLU decisions inside the band where fp32 accumulation (and the
    # layer's stored input, compared below) leaves the sign open follow the
    # GPU, whose value there must be that small
    hs_ref, _ = omlp.mlp_forward(x, layers, rnd, relu_last)
    ov = []
    for i, (W, b) in enumerate(layers):
        if i == len(layers) - 1 and not relu_last:
            ov.append(None)
            continue
        a = omlp.linear(hs_ref[i], W, b)
        band = omlp.relu_band(hs_ref[i], W, b)
        if i > 0:
            h_gpu = acts[i - 1].float().cpu().double().numpy()
            band = band + np.abs(h_gpu - hs_ref[i]) @ np.abs(np.asarray(W, np.float64)).T
        where = np.abs(a) <= band
        out_gpu = acts[i].float().cpu().double().numpy()
        assert np.all(np.abs(out_gpu[where]) <= 2.01 * band[where] + 1e-30), f"layer {i}: GPU value outside band"
        ov.append((where, out_gpu > 0))
    hs, masks = omlp.mlp_forward(x, layers, rnd, relu_last, overrides=ov)
    for i in range(len(layers)):
        assert_close(f"act{i}", acts[i], hs[i + 1], t)
    if relu_last:
        g_out_np = synth.randn((B, dims[-1]), seed=13, scale=1e-2, dtype=dt)
        g_out = to_dev(g_out_np, sdt)
    else:
        lval, dz = oloss.masked_bce(hs[-1], y, m)
        assert_close("loss", loss["loss"], np.array([lval]), t)
        assert_close("d_logits", loss["d_logits"], dz, t)
        g_out_np = rnd(dz)
        g_out = loss["d_logits_op"]
    d_in = torch.zeros((B, dims[0]), dtype=sdt, device=DEV)
    api.lattice_mlp_heads_bwd(L, xd, acts, g_out, relu_last, d_in=d_in)
    torch.cuda.synchronize()
    dWs, dbs, dh0 = omlp.mlp_backward(g_out_np, hs, masks, layers, rnd, relu_last, need_input_grad=True)
    for i in range(len(layers)):
        assert_close(f"dW{i}", L[i]["dW"], dWs[i], t)
        assert_close(f"db{i}", L[i]["db"], dbs[i], t)
    assert_close("d_in", d_in, rnd(dh0), t)
