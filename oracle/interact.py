"""Feature interaction over the stacked per-sample vectors X_b (n x d, one row
per vector).

Test infrastructure only (see the package docstring).

* DOT (pairwise dot products; the DLRM-style interaction used as a baseline
  in Section 4):  ``p[b, m(i,j)] = <X_b[i], X_b[j]>`` for ``0 <= i < j < n`` in
  row-major order of the strict upper triangle,
  ``m(i,j) = i*n - i*(i+1)/2 + (j-i-1)``.  Backward: with the symmetric matrix
  ``S`` holding ``dp`` at (i,j) and (j,i) and a zero diagonal,
  ``dX_b = S X_b``.
* FM (the factorization-machine block of the DHEN/Wukong fusion block,
  Section 3.3.2): ``O_b = X_b (X_b^T W)`` with ``W`` of shape n x k, i.e. the
  n x n Gram matrix ``X_b X_b^T`` projected onto k columns without ever forming
  it.  Storage points: ``P_b = rnd(X_b^T W)`` (d x k), ``O_b = rnd(X_b P_b)``.
  Backward given ``G_b = dO_b``: ``dP_b = rnd(X_b^T G_b)``,
  ``dX_b = G_b P_b^T + W dP_b^T``, ``dW = sum_b X_b dP_b``.
* STACK: L layers of [FM block (rank k) -> linear compression of vec(F) back
  to n_out vectors of dim d (no bias: the backbone is bias-less, Section
  3.3.4) -> + residual (identity, or a linear compression block ``C X`` when
  the vector count changes) -> LayerNorm over d with gain only (bias-less,
  computed at fp32 or better, Section 3.5.2)], each output stored as
  ``rnd(...)``.
"""
import numpy as np


def pair_indices(n):
    """(i, j) of the strict upper triangle in row-major order."""
    return np.triu_indices(n, k=1)


def dot_forward(X, rnd):
    X = np.asarray(X, np.float64)
    Z = X @ X.transpose(0, 2, 1)
    i, j = pair_indices(X.shape[1])
    return rnd(Z[:, i, j])


def dot_backward(dp, X):
    X = np.asarray(X, np.float64)
    B, n, _ = X.shape
    i, j = pair_indices(n)
    S = np.zeros((B, n, n), dtype=np.float64)
    S[:, i, j] = dp
    S[:, j, i] = dp
    return S @ X


def fm_forward(X, W, rnd):
    """(O [B,n,k], P [B,d,k])."""
    X = np.asarray(X, np.float64)
    W = np.asarray(W, np.float64)
    P = rnd(X.transpose(0, 2, 1) @ W)
    O = rnd(X @ P)
    return O, P


def fm_backward(G, X, W, P, rnd):
    """(dX [B,n,d] float64, dW [n,k]) given G = dO (already at storage precision)."""
    G = np.asarray(G, np.float64)
    X = np.asarray(X, np.float64)
    W = np.asarray(W, np.float64)
    dP = rnd(X.transpose(0, 2, 1) @ G)                      # [B, d, k]
    dX = G @ P.transpose(0, 2, 1) + W[None] @ dP.transpose(0, 2, 1)
    dW = (X @ dP).sum(axis=0)
    return dX, dW


def layernorm_forward(u, gamma, eps):
    """Per-vector LayerNorm over the last axis, gain only (population variance)."""
    u = np.asarray(u, np.float64)
    mu = u.mean(axis=-1, keepdims=True)
    var = ((u - mu) ** 2).mean(axis=-1, keepdims=True)
    rstd = 1.0 / np.sqrt(var + eps)
    xhat = (u - mu) * rstd
    return np.asarray(gamma, np.float64) * xhat, xhat, rstd


def layernorm_backward(dy, xhat, rstd, gamma):
    """(du, dgamma)."""
    dy = np.asarray(dy, np.float64)
    dgamma = (dy * xhat).reshape(-1, xhat.shape[-1]).sum(axis=0)
    dxh = dy * np.asarray(gamma, np.float64)
    du = rstd * (dxh - dxh.mean(axis=-1, keepdims=True)
                 - xhat * (dxh * xhat).mean(axis=-1, keepdims=True))
    return du, dgamma


def stack_forward(X1, layers, n_out, d, rnd, eps, fp8=False):
    """Returns (X_{L+1}, per-layer caches).  A layer with an ``L`` matrix
    ([n_lcb, n_in]) is a full fusion block: its FM block fills the first
    ``n_out - n_lcb`` output vectors and the linear compression block
    ``L X`` the last ``n_lcb`` (concatenated before the residual and the
    LayerNorm).  fp8: the FM block's projection vec(F) A^T as an FP8 linear
    layer (Section 3.5.2: linear layers in FP8 with row-wise scales): vec(F)
    quantised per sample and A per output unit (oracle.fp8.quantize), the
    product of the codes times both scales (oracle.fp8.linear_fp8)."""
    from oracle import fp8 as ofp8
    X = np.asarray(X1, np.float64)
    B = X.shape[0]
    caches = []
    for lay in layers:
        Fm, P = fm_forward(X, lay["W"], rnd)                  # [B, n, k]
        vecF = Fm.reshape(B, -1)
        if fp8:
            qf, sf = ofp8.quantize(vecF, rowwise=True)
            qa, sa = ofp8.quantize(np.asarray(lay["A"], np.float64), rowwise=True)
            HF = ofp8.linear_fp8(qf, sf, qa, sa).reshape(B, -1, d)
        else:
            HF = (vecF @ np.asarray(lay["A"], np.float64).T).reshape(B, -1, d)
        if lay.get("L") is not None:
            HL = np.einsum("vu,bud->bvd", np.asarray(lay["L"], np.float64), X)
            H = np.concatenate([HF, HL], axis=1)
        else:
            H = HF
        assert H.shape[1] == n_out
        if lay.get("C") is not None:
            res = np.einsum("vu,bud->bvd", np.asarray(lay["C"], np.float64), X)
        else:
            res = X
        y, xhat, rstd = layernorm_forward(H + res, lay["gamma"], eps)
        caches.append(dict(X=X, P=P, vecF=vecF, xhat=xhat, rstd=rstd))
        X = rnd(y)
    return X, caches


def stack_backward(dY, layers, caches, rnd):
    """Backward through ``stack_forward`` given dY = dL/dX_{L+1}.
    Returns (dX_1 float64, per-layer grads dict list)."""
    dY = np.asarray(dY, np.float64)
    grads = [None] * len(layers)
    for li in range(len(layers) - 1, -1, -1):
        lay, c = layers[li], caches[li]
        X = c["X"]
        B, n, _ = X.shape
        du, dgamma = layernorm_backward(dY, c["xhat"], c["rstd"], lay["gamma"])
        duR = rnd(du)
        A = np.asarray(lay["A"], np.float64)
        nF = A.shape[0] // du.shape[2]                       # FM-block output vectors
        du2 = duR[:, :nF].reshape(B, -1)
        dA = du2.T @ c["vecF"]
        dF = rnd((du2 @ A).reshape(B, n, -1))
        dX, dW = fm_backward(dF, X, lay["W"], c["P"], rnd)
        g = dict(dW=dW, dA=dA, dgamma=dgamma)
        if lay.get("L") is not None:
            Lm = np.asarray(lay["L"], np.float64)
            g["dL"] = np.einsum("bvd,bud->vu", duR[:, nF:], X)
            dX = dX + np.einsum("vu,bvd->bud", Lm, duR[:, nF:])
        if lay.get("C") is not None:
            C = np.asarray(lay["C"], np.float64)
            g["dC"] = np.einsum("bvd,bud->vu", duR, X)
            dX = dX + np.einsum("vu,bvd->bud", C, duR)
        else:
            dX = dX + du
        grads[li] = g
        dY = dX
    return dY, grads
