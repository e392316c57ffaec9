"""Per-objective towers through the C ABI's MLP entry points (Section
3.3.3): a tower layer of T groups of H units, then the grouped heads
(objective t reads only group t), forward and backward, each stage against
the oracle on the GPU's own stored inputs of that stage."""
import numpy as np
import pytest
import torch

from oracle import mlp as omlp
from tests._util import DEV, _np64, assert_product

CASES = [
    # B, K, T, H, dtype
    (300, 200, 6, 16, "bf16"),      # ragged rows and K
    (1024, 512, 16, 32, "bf16"),
    (5, 24, 3, 8, "bf16"),
    (257, 100, 4, 24, "f32"),
]


@pytest.mark.gpu
@pytest.mark.parametrize("B,K,T,H,dtype", CASES)
def test_tower_heads(B, K, T, H, dtype):
    from paper_2512_09200_amd import api
    print(f"[towers] B={B} K={K} T={T} H={H} {dtype}", flush=True)
    rng = np.random.default_rng(B + 7 * T)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    dev = lambda a, dt=tdt: torch.from_numpy(np.asarray(a, np.float32)).to(dt).to(DEV)
    x = dev(rng.standard_normal((B, K)))
    W0 = dev(rng.standard_normal((T * H, K)) / np.sqrt(K))
    W1 = dev(rng.standard_normal((T, H)) / np.sqrt(H))
    b0, b1 = dev(0.1 * rng.standard_normal(T * H), torch.float32), dev(0.1 * rng.standard_normal(T), torch.float32)
    z32 = lambda *s: torch.zeros(*s, device=DEV)
    layers = [dict(W=W0, b=b0, dW=z32(T * H, K), db=z32(T * H)), dict(W=W1, b=b1, dW=z32(T, H), db=z32(T))]
    h1 = torch.zeros(B, T * H, dtype=tdt, device=DEV)
    z = torch.zeros(B, T, device=DEV)
    api.lattice_mlp_heads_fwd(layers, x, [h1, z], relu_last=False, tower_heads=True)
    d_out = dev(rng.standard_normal((B, T)))
    d_in = torch.zeros(B, K, dtype=tdt, device=DEV)
    api.lattice_mlp_heads_bwd(layers, x, [h1, z], d_out, relu_last=False, d_in=d_in, tower_heads=True)
    torch.cuda.synchronize()
    us = 2.0 ** -8 if dtype == "bf16" else None
    t = 2e-2 if dtype == "bf16" else 1e-5
    X, A0, A1, B0, B1 = (_np64(v) for v in (x, W0, W1, b0, b1))
    H1, G = _np64(h1), _np64(d_out)
    a = X @ A0.T + B0
    assert_product("tower layer", H1, np.maximum(a, 0), np.abs(X) @ np.abs(A0).T + np.abs(B0), K + 1, us, t)
    assert_product("logits", z, omlp.grouped_linear(H1, A1, B1),
                   omlp.grouped_linear(np.abs(H1), np.abs(A1), np.abs(B1)), H + 1, None, t)
    dW1, db1, dh = omlp.grouped_linear_grads(G, H1, A1)
    adW1, adb1, adh = omlp.grouped_linear_grads(np.abs(G), np.abs(H1), np.abs(A1))
    assert_product("heads dW", layers[1]["dW"], dW1, adW1, B, None, t)
    assert_product("heads db", layers[1]["db"], db1, adb1, B, None, t)
    # the tower layer's pre-activation gradient (masked by its ReLU), as the
    # GPU stores it, then the tower layer's gradients and the input gradient
    on = H1 > 0
    gh = dh * on
    gh_s = gh if us is None else np.asarray(torch.from_numpy(gh).to(torch.bfloat16).double().numpy())
    assert_product("tower dW", layers[0]["dW"], gh_s.T @ X, np.abs(gh_s).T @ np.abs(X), B, None, t)
    assert_product("tower db", layers[0]["db"], gh_s.sum(0), np.abs(gh_s).sum(0), B, None, t)
    assert_product("d_in", d_in, gh_s @ A0, np.abs(gh_s) @ np.abs(A0), T * H, us, t)
