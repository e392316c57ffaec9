"""A dense layer whose input spans more than 2 GiB (66000 x 16384 bf16): the
GEMMs whose operands do not fit a 2 GiB buffer resource take the per-load
pointer loaders (forward, and the weight gradient whose M-contiguous B is
that input), the input gradient the buffer loaders with a k-major weight
operand.  One ReLU layer (Section 3.3.1's MLP layers) forward and backward
through the C ABI; every stage recomputed by the oracle from the
accelerator's own stored operands on sampled rows and columns (all of the
bias gradient)."""
import numpy as np
import pytest
import torch

from tests._util import DEV, _np64, assert_product

B, K, N = 66000, 16384, 256


@pytest.mark.gpu
def test_layer_with_input_over_2gib():
    from paper_2512_09200_amd import api
    assert B * K * 2 > 2 ** 31
    print(f"[gemm-large] B={B} K={K} N={N} (input {B * K * 2 / 2**30:.2f} GiB)", flush=True)
    g = torch.Generator(device=DEV).manual_seed(2512)
    x = torch.empty((B, K), dtype=torch.bfloat16, device=DEV)
    for r0 in range(0, B, 8192):
        r1 = min(B, r0 + 8192)
        x[r0:r1] = torch.randn((r1 - r0, K), device=DEV, generator=g).to(torch.bfloat16)
    W = (torch.randn((N, K), device=DEV, generator=g) / np.sqrt(K)).to(torch.bfloat16)
    b = 0.01 * torch.randn(N, device=DEV, generator=g)
    L = [dict(W=W, b=b, dW=torch.zeros((N, K), device=DEV), db=torch.zeros(N, device=DEV))]
    y = torch.empty((B, N), dtype=torch.bfloat16, device=DEV)
    api.lattice_mlp_heads_fwd(L, x, [y], True)
    torch.cuda.synchronize()
    rng = np.random.default_rng(7)
    rows = np.unique(np.concatenate([rng.choice(B, 62, replace=False), [0, B - 1]]))
    ri = torch.from_numpy(rows).to(DEV)
    X = _np64(x[ri])
    Wn, bn = _np64(W), _np64(b)
    a = X @ Wn.T + bn
    absa = np.abs(X) @ np.abs(Wn).T + np.abs(bn)
    us = 2.0 ** -8
    assert_product("forward (sampled rows)", y[ri], np.maximum(a, 0), absa, K + 1, us)

    # backward from a random output gradient; the ReLU mask is the GPU's own output
    gout = (0.01 * torch.randn((B, N), device=DEV, generator=g)).to(torch.bfloat16)
    d_in = torch.empty((B, K), dtype=torch.bfloat16, device=DEV)
    api.lattice_mlp_heads_bwd(L, x, [y], gout, True, d_in=d_in)
    torch.cuda.synchronize()
    # the pre-activation gradient as the GPU forms it (bf16 operand of the products)
    dpre = (gout.float() * (y.float() > 0)).to(torch.bfloat16)
    cols = np.unique(np.concatenate([rng.choice(K, 30, replace=False), [0, K - 1]]))
    ci = torch.from_numpy(cols).to(DEV)
    Dp = _np64(dpre)
    Xc = _np64(x[:, ci])
    assert_product("dW (sampled columns)", L[0]["dW"][:, ci], Dp.T @ Xc, np.abs(Dp).T @ np.abs(Xc), B)
    assert_product("db", L[0]["db"], Dp.sum(0), np.abs(Dp).sum(0), B)
    Dr = Dp[rows]
    assert_product("d_in (sampled rows)", d_in[ri], Dr @ Wn, np.abs(Dr) @ np.abs(Wn), N, us)
    del x, d_in
    torch.cuda.empty_cache()
