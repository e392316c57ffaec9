"""One forward + backward training step of the sparse-dense core, composed
from the plain definitions in this package.

Test infrastructure only (see the package docstring).

Forward (per sample b; Section 3.3):
  1. pooled embeddings of every categorical feature -> slots
     ``first_slot .. first_slot+F-1`` of the stacked X_b (Section 3.3.1);
  2. dense features through the bottom MLP (ReLU on every layer) -> slot 0;
  3. interaction (DOT, FM or STACK, see ``interact``);
  4. top input: ``concat(X_b[0], flatten(interaction))`` (DOT/FM), or the
     flattened STACK output;
  5. top MLP, ReLU (or SwishRN, Section 3.3.4) on hidden layers, one logit
     per objective (Section 3.3.3; with towers the last hidden layer holds
     one group of units per objective and each logit reads only its group;
     untied layers use the parameter set of the sample's domain, Section
     3.3.4);
  6. masked BCE (Section 3.2.1).
Backward: the exact chain rule through 1-6, with GEMM operands (activation
gradients) rounded to the storage precision where the accelerator stores them:
the logit gradient, every hidden-activation gradient, the gradient of the top
input, the FM/STACK intermediate gradients, and the gradient of the embedding
slots (the input of the sparse gradient).  Weight gradients are not rounded.
"""
import numpy as np

from . import bf16 as _bf16
from .embbag import pool_forward, pool_backward, bookkeeping, sgd_rows
from .mlp import mlp_forward, mlp_backward
from .interact import (dot_forward, dot_backward, fm_forward, fm_backward,
                       stack_forward, stack_backward)
from .loss import masked_bce


def rounding(dtype):
    """Storage rounding of a workload: bf16 RNE, or none for fp32."""
    return _bf16.round_bf16 if dtype == "bf16" else _bf16.identity


def top_act(cfg, params):
    """The SwishRN description of the top MLP's hidden layers (see
    ``mlp.mlp_forward``), or None for ReLU."""
    if getattr(cfg, "top_act", "relu") == "relu":
        return None
    kind = {"swishrn": "sigmoid", "hardswishrn": "hard"}[cfg.top_act]
    return dict(kind=kind, block=cfg.norm_block, eps=cfg.norm_eps, gains=params["top_gain"])


def forward(cfg, params, table, batch, overrides=None, loss_normalizer=None, fp8_top=False):
    """``overrides`` (optional) maps "bottom"/"top" to per-layer ReLU decision
    overrides (see ``mlp.mlp_forward``) and "top_gate" to per-layer hard-gate
    derivative overrides of the backward (see ``swishrn.backward``); ``loss_normalizer`` (optional) is the
    labelled-entry count of the full batch when ``batch`` holds a subset of
    its samples.  ``fp8_top``: the top MLP's hidden layers run their forward
    product in FP8 with row-wise scales (mixed FP8 / BF16 training, Section
    3.5.2); the objective heads and the whole backward keep the stored bf16
    values (the gradient treats quantisation as the identity)."""
    rnd = rounding(cfg.dtype)
    B, F, d = int(cfg.B), int(cfg.F), int(cfg.d)
    n, s0 = cfg.n_slots, cfg.first_emb_slot
    c = {}
    pooled = pool_forward(table, batch["row_base"], batch["offsets"], batch["indices"], F, B, cfg.pool)
    X = np.zeros((B, n, d), dtype=np.float64)
    X[:, s0:] = rnd(pooled)
    if cfg.has_dense:
        hs, mb = mlp_forward(batch["dense"], params["bottom"], rnd, relu_last=True,
                         overrides=(overrides or {}).get("bottom"))
        X[:, 0] = hs[-1]
        c["hs_bottom"], c["masks_bottom"] = hs, mb
    c["X"] = X
    head = [X[:, 0]] if cfg.has_dense else []
    if cfg.interact == "dot":
        inter = dot_forward(X, rnd)
        t = np.concatenate(head + [inter], axis=1)
    elif cfg.interact == "fm":
        O, P = fm_forward(X, params["fm_W"], rnd)
        c["fm_P"] = P
        inter = O.reshape(B, -1)
        t = np.concatenate(head + [inter], axis=1)
    elif cfg.interact == "stack":
        XL, caches = stack_forward(X, params["stack"], cfg.stack_n, d, rnd, cfg.ln_eps)
        c["stack"] = caches
        inter = XL.reshape(B, -1)
        t = inter
    else:
        raise ValueError(cfg.interact)
    c["inter"] = inter
    hs_top, mt = mlp_forward(t, params["top"], rnd, relu_last=False,
                         overrides=(overrides or {}).get("top"),
                         fp8_layers=tuple(range(len(params["top"]) - 1)) if fp8_top else (),
                         act=top_act(cfg, params), grouped_last=bool(getattr(cfg, "towers", 0)),
                         domain=batch.get("domain"))
    c["hs_top"], c["masks_top"] = hs_top, mt
    c["gate_overrides"] = (overrides or {}).get("top_gate")
    z = hs_top[-1]
    loss, dz = masked_bce(z, batch["labels"], batch["mask"], loss_normalizer)
    c.update(logits=z, loss=loss, dz=dz, t=t)
    return c


def backward(cfg, params, table, batch, c, lr_tables=None):
    rnd = rounding(cfg.dtype)
    B, F, d = int(cfg.B), int(cfg.F), int(cfg.d)
    s0 = cfg.first_emb_slot
    X = c["X"]
    g = {}
    gz = rnd(c["dz"])
    act = top_act(cfg, params)
    if act is not None:
        act["overrides"] = c.get("gate_overrides")
    dgains = [None] * (len(params["top"]) - 1)
    dWt, dbt, dt = mlp_backward(gz, c["hs_top"], c["masks_top"], params["top"], rnd, relu_last=False,
                                need_input_grad=True, act=act, dgains=dgains,
                                grouped_last=bool(getattr(cfg, "towers", 0)), domain=batch.get("domain"))
    g["top_dW"], g["top_db"] = dWt, dbt
    if act is not None:
        g["top_dgain"] = dgains
    gt = rnd(dt)
    g["d_top_in"] = gt
    off = d if cfg.has_dense else 0
    if cfg.interact == "dot":
        dXi = dot_backward(gt[:, off:], X)
    elif cfg.interact == "fm":
        G = gt[:, off:].reshape(B, cfg.n_slots, cfg.fm_rank)
        dXi, dWfm = fm_backward(G, X, params["fm_W"], c["fm_P"], rnd)
        g["fm_dW"] = dWfm
    else:
        dXi, sg = stack_backward(gt.reshape(B, cfg.stack_n, d), params["stack"], c["stack"], rnd)
        g["stack"] = sg
    dX_emb = rnd(dXi[:, s0:])
    g["dX_emb"] = dX_emb
    if cfg.has_dense:
        dh = dXi[:, 0] + gt[:, :d]
        dWb, dbb, _ = mlp_backward(dh, c["hs_bottom"], c["masks_bottom"], params["bottom"], rnd, relu_last=True,
                                   need_input_grad=False)
        g["bottom_dW"], g["bottom_db"] = dWb, dbb
    uniq, G = pool_backward(dX_emb, batch["row_base"], batch["offsets"], batch["indices"], F, B, cfg.pool)
    g["unique_rows"], g["grad_rows"] = uniq, G
    g["bookkeeping"] = bookkeeping(batch["row_base"], batch["offsets"], batch["indices"], F, B)
    lr = cfg.lr_tables if lr_tables is None else lr_tables
    if lr:
        g["updated_rows"] = sgd_rows(np.asarray(table, np.float64)[uniq], G, lr, rnd)
    return g


def step(cfg, params, table, batch, lr_tables=None, overrides=None, loss_normalizer=None, fp8_top=False):
    c = forward(cfg, params, table, batch, overrides, loss_normalizer, fp8_top)
    g = backward(cfg, params, table, batch, c, lr_tables)
    return c, g
