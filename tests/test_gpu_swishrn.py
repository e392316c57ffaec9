"""SwishRN layers on the GPU (Sections 3.3.4 and 3.5.3) through the C ABI's
MLP entry points: the BlockNorm statistic in the bf16 GEMM's epilogue (128-
and 256-column tiles), the unfused path (whole-row RMSNorm, fp32 models),
both gates, ragged rows, widths and groups, and the backward (chain, weight
and gain gradients) -- each against the oracle on the GPU's own stored
inputs of that stage, within the derived fp32 bounds."""
import numpy as np
import pytest
import torch

from oracle import swishrn as oswish
from tests._util import (DEV, _np64, assert_bounded, check_swishrn_forward, check_swishrn_gains)

U = 2.0 ** -24

CASES = [
    # B, K, N, dtype, block, act
    (300, 200, 200, "bf16", 128, "swishrn"),       # ragged rows, K and last group (72)
    (300, 200, 200, "bf16", 0, "hardswishrn"),     # whole-row RMSNorm: GEMM, then the row kernel
    (64, 64, 1024, "bf16", 128, "hardswishrn"),
    (1, 32, 130, "bf16", 128, "swishrn"),          # one row; a group of 2
    (8192, 256, 2048, "bf16", 128, "swishrn"),     # 256x256 tiles: two groups per tile
    (8192, 256, 2048, "bf16", 128, "hardswishrn"),
    (257, 100, 300, "f32", 128, "swishrn"),        # fp32: BlockNorm groups in the row kernel
    (257, 100, 300, "f32", 0, "hardswishrn"),
]


def _kind(act):
    return "sigmoid" if act == "swishrn" else "hard"


def _layer(B, K, N, dtype, block, seed):
    rng = np.random.default_rng(seed)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    x = torch.from_numpy(rng.standard_normal((B, K)).astype(np.float32)).to(tdt).to(DEV)
    W = torch.from_numpy((rng.standard_normal((N, K)) / np.sqrt(K)).astype(np.float32)).to(tdt).to(DEV)
    b = torch.from_numpy((0.1 * rng.standard_normal(N)).astype(np.float32)).to(DEV)
    gain = torch.from_numpy((1 + 0.25 * rng.standard_normal((2, N))).astype(np.float32)).to(DEV)
    groups = 1 if block <= 0 or block >= N else -(-N // block)
    L = dict(W=W, b=b, gain=gain, dW=torch.zeros(N, K, device=DEV), db=torch.zeros(N, device=DEV),
             dgain=torch.zeros(2, N, device=DEV), pre=torch.zeros(B, N, dtype=tdt, device=DEV),
             rinv=torch.zeros(B, groups, device=DEV))
    d_out = torch.from_numpy(rng.standard_normal((B, N)).astype(np.float32)).to(tdt).to(DEV)
    return x, L, d_out


@pytest.mark.gpu
@pytest.mark.parametrize("B,K,N,dtype,block,act", CASES)
def test_swishrn_layer(B, K, N, dtype, block, act):
    from paper_2512_09200_amd import api
    print(f"[swishrn] B={B} K={K} N={N} {dtype} block={block} {act}", flush=True)
    x, L, d_out = _layer(B, K, N, dtype, block, seed=B * 7 + N)
    out = torch.zeros(B, N, dtype=x.dtype, device=DEV)
    eps = 1e-6
    api.lattice_mlp_heads_fwd([L], x, [out], relu_last=True, act=act, norm_block=block, norm_eps=eps)
    d_in = torch.zeros(B, K, dtype=x.dtype, device=DEV)
    api.lattice_mlp_heads_bwd([L], x, [out], d_out, relu_last=True, d_in=d_in, act=act,
                              norm_block=block, norm_eps=eps)
    torch.cuda.synchronize()
    us = 2.0 ** -8 if dtype == "bf16" else None
    t = 2e-2 if dtype == "bf16" else 1e-5
    gains = _np64(L["gain"])
    oact = dict(kind=_kind(act), block=block, eps=eps, gains=[(gains[0], gains[1])])
    h, W, b = _np64(x), _np64(L["W"]), _np64(L["b"])

    class _Cfg:
        pass
    cfg = _Cfg()
    cfg.dtype = dtype
    check_swishrn_forward("layer", cfg, oact, 0, h, W, b, _np64(L["pre"]), _np64(L["rinv"]), out, us, t)
    # backward from the stored d_out, pre-activation and rho
    check_swishrn_gains("layer", oact, 0, d_out, L["pre"], L["rinv"], L["dgain"], t)
    go, pre, rinv = _np64(d_out), _np64(L["pre"]), _np64(L["rinv"])
    dh, _, _ = oswish.backward(go, pre, gains[0], gains[1], block, eps, _kind(act), rho=rinv)
    e_dh, _, _ = oswish.backward_bound(go, 0.0, pre, gains[0], gains[1], block, eps, _kind(act), rinv)
    # the chain's value reaches the products through its storage rounding
    e_g = e_dh + (us * (np.abs(dh) + e_dh) if us else 0.0)
    ag = np.abs(dh) + e_g
    assert_bounded("d_in", d_in, dh @ W, e_g @ np.abs(W) + (N + 3) * U * (ag @ np.abs(W)), us, t)
    assert_bounded("dW", L["dW"], dh.T @ h, e_g.T @ np.abs(h) + (B + 3) * U * (ag.T @ np.abs(h)), None, t)
    assert_bounded("db", L["db"], dh.sum(0), e_g.sum(0) + (B + 3) * U * ag.sum(0), None, t)


@pytest.mark.gpu
def test_swishrn_empty_batch_zero_gradients():
    from paper_2512_09200_amd import api
    x, L, d_out = _layer(0, 64, 128, "bf16", 128, seed=1)
    for k in ("dW", "db", "dgain"):
        L[k].fill_(7.0)
    api.lattice_mlp_heads_fwd([L], x, [torch.zeros(0, 128, dtype=x.dtype, device=DEV)], relu_last=True,
                              act="swishrn")
    api.lattice_mlp_heads_bwd([L], x, [torch.zeros(0, 128, dtype=x.dtype, device=DEV)], d_out,
                              relu_last=True, act="swishrn")
    torch.cuda.synchronize()
    for k in ("dW", "db", "dgain"):
        assert torch.count_nonzero(L[k]).item() == 0, k
