"""Seeded synthetic inputs for the sparse-dense training step.

This module draws random numbers and lays them out; it holds none of the
method's arithmetic.  Both the HIP path (tests, benchmark) and the CPU oracle
take their inputs from here.

Recipe (stated once, used everywhere):

* Every tensor has its own stream: ``numpy.random.default_rng([seed, stream,
  batch_id])`` (PCG64), so batches and parameters are reproducible and
  independent of one another.
* Jagged categorical batch in feature-major layout: bag ``f*B + b`` holds the
  indices of feature ``f`` for sample ``b``; ``offsets`` has ``F*B+1`` int32
  entries and ``indices`` holds table-local row ids (int32).
* Bag lengths: discrete uniform, or Poisson clipped to ``[lo, hi]``.  In the
  multi-domain workload a feature that the sample's domain does not activate
  has an empty bag (zero-padding of missing features in the unified dataset,
  Section 3.2).
* Indices: uniform over rows, or a bounded Zipf law ``P(k) ~ k^-alpha`` for
  rank ``k = 1..N`` drawn by inverse CDF in fp64; rank ``k`` maps to row
  ``((k-1)*A_f + C_f) mod N`` with ``gcd(A_f, N) = 1`` so hot rows are
  scattered through the table as hashed ids would be.
* Tables: N(0, 0.01^2), drawn per table with ``torch.randn`` on the target
  device (seed derived from the config seed and the table id).
* Linear weights ``[out, in]``: Glorot normal N(0, 2/(in+out)); biases
  N(0, 0.01^2); FM projection ``W [n, k]``: N(0, 1/n); LayerNorm gain
  ``1 + N(0, 0.1^2)``.
* Dense inputs N(0, 1).  Labels Bernoulli(p_t) with p_t fixed or drawn per
  objective from U[lo, hi].  Mask: all ones, i.i.d. Bernoulli(keep), or per
  domain (each domain labels a seeded subset of the objectives).
* bf16 workloads store tables, dense inputs and weights in bf16
  (round-to-nearest-even from fp32, done by torch); biases and gains stay fp32.
"""
from __future__ import annotations

import math
from typing import Dict, List, Optional

import numpy as np
import torch

from .configs import Config

# stream ids (arbitrary, fixed)
_S_BAGLEN, _S_INDEX, _S_DENSE, _S_LABEL_P, _S_LABEL, _S_MASK = 1, 2, 3, 4, 5, 6
_S_DOMAIN, _S_PERM = 7, 8
_S_BOTTOM, _S_TOP, _S_FM, _S_STACK, _S_TABLE, _S_GAIN, _S_TOWER, _S_UNTIE = 20, 21, 22, 23, 24, 25, 26, 27
_S_AUX = 40


def _rng(seed: int, stream: int, sub: int = 0) -> np.random.Generator:
    return np.random.default_rng([int(seed), int(stream), int(sub)])


def torch_dtype(name: str) -> torch.dtype:
    return {"f32": torch.float32, "bf16": torch.bfloat16}[name]


def to_storage(x: np.ndarray, dtype: str, device="cpu") -> torch.Tensor:
    """fp64/fp32 numpy array -> torch tensor in the storage dtype (RNE)."""
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch_dtype(dtype)).to(device)


# ---------------------------------------------------------------------------
# index distributions
# ---------------------------------------------------------------------------
_ZIPF_CACHE: Dict = {}


def zipf_cdf(N: int, alpha: float) -> np.ndarray:
    key = (N, alpha)
    if key not in _ZIPF_CACHE:
        k = np.arange(1, N + 1, dtype=np.float64)
        c = np.cumsum(k ** (-alpha))
        _ZIPF_CACHE[key] = c / c[-1]
    return _ZIPF_CACHE[key]


def zipf_ranks(rng: np.random.Generator, N: int, alpha: float, size: int) -> np.ndarray:
    """Ranks in 1..N with P(k) proportional to k^-alpha (inverse CDF, fp64)."""
    u = rng.random(size)
    return np.searchsorted(zipf_cdf(N, alpha), u, side="right").astype(np.int64) + 1


def rank_permutation(seed: int, f: int, N: int):
    """(A, C) of the bijection rank k -> ((k-1)*A + C) mod N for table f."""
    r = _rng(seed, _S_PERM, f)
    while True:
        A = int(r.integers(1, max(2, N)))
        if math.gcd(A, N) == 1:
            break
    C = int(r.integers(0, N))
    return A, C


# ---------------------------------------------------------------------------
# batch
# ---------------------------------------------------------------------------
def _domain_plan(cfg: Config):
    """Per-domain active-feature sets and labelled heads (seeded)."""
    props, n_active, n_heads = cfg.domains
    r = _rng(cfg.seed, _S_DOMAIN, 0)
    feats = [np.sort(r.choice(cfg.F, size=n_active, replace=False)) for _ in props]
    heads = [np.sort(r.choice(cfg.T, size=n_heads, replace=False)) for _ in props]
    return props, feats, heads


def domain_counts(B: int, props) -> List[int]:
    """Exact per-domain sample counts by largest remainder."""
    raw = [p * B for p in props]
    base = [int(math.floor(x)) for x in raw]
    rem = B - sum(base)
    order = sorted(range(len(props)), key=lambda i: (-(raw[i] - base[i]), i))
    for i in order[:rem]:
        base[i] += 1
    return base


def make_batch(cfg: Config, batch_id: int = 0) -> Dict[str, np.ndarray]:
    """One synthetic batch as numpy arrays (host memory)."""
    B, F, N = cfg.B, cfg.F, cfg.rows
    seed = cfg.seed

    # ---- domains / activity ----
    domain = np.zeros(B, dtype=np.uint8)
    active = np.ones((F, B), dtype=bool)
    mask = np.ones((B, cfg.T), dtype=np.uint8)
    if cfg.mask[0] == "domain":
        props, feats, heads = _domain_plan(cfg)
        counts = domain_counts(B, props)
        dom = np.concatenate([np.full(c, i, dtype=np.uint8) for i, c in enumerate(counts)])
        if not cfg.untie:
            _rng(seed, _S_DOMAIN, 1000 + batch_id).shuffle(dom)
        # (untied parameters: samples grouped by domain, in domain order)
        domain = dom
        active[:] = False
        mask[:] = 0
        for i in range(len(props)):
            sel = domain == i
            for f in feats[i]:
                active[f, sel] = True
            for t in heads[i]:
                mask[sel, t] = 1
    elif cfg.mask[0] == "iid":
        keep = cfg.mask[1]
        mask = (_rng(seed, _S_MASK, batch_id).random((B, cfg.T)) < keep).astype(np.uint8)

    # ---- bag lengths ----
    r = _rng(seed, _S_BAGLEN, batch_id)
    kind = cfg.bag_dist[0]
    if kind == "uniform":
        lens = r.integers(cfg.bag_dist[1], cfg.bag_dist[2] + 1, size=(F, B))
    elif kind == "poisson":
        lens = np.clip(r.poisson(cfg.bag_dist[1], size=(F, B)), cfg.bag_dist[2], cfg.bag_dist[3])
    else:
        raise ValueError(kind)
    lens = np.where(active, lens, 0).astype(np.int64)
    offsets = np.zeros(F * B + 1, dtype=np.int64)
    np.cumsum(lens.reshape(-1), out=offsets[1:])
    nnz = int(offsets[-1])
    if nnz >= 2**31:
        raise ValueError("nnz does not fit int32")

    # ---- indices (per feature, so the rank permutation is per table) ----
    indices = np.empty(nnz, dtype=np.int32)
    for f in range(F):
        lo, hi = int(offsets[f * B]), int(offsets[(f + 1) * B])
        m = hi - lo
        if m == 0:
            continue
        ri = _rng(seed, _S_INDEX, batch_id * 65536 + f)
        if cfg.index_dist[0] == "uniform":
            indices[lo:hi] = ri.integers(0, N, size=m)
        else:
            k = zipf_ranks(ri, N, cfg.index_dist[1], m)
            A, C = rank_permutation(seed, f, N)
            indices[lo:hi] = (((k - 1) * A + C) % N).astype(np.int32)

    # ---- dense, labels ----
    dense = _rng(seed, _S_DENSE, batch_id).standard_normal((B, cfg.dense_in)).astype(np.float32)
    if cfg.dtype == "bf16":
        dense = to_storage(dense, "bf16").float().numpy()
    if cfg.label_p[0] == "fixed":
        p = np.full(cfg.T, cfg.label_p[1])
    else:
        p = _rng(seed, _S_LABEL_P, 0).uniform(cfg.label_p[1], cfg.label_p[2], size=cfg.T)
    labels = (_rng(seed, _S_LABEL, batch_id).random((B, cfg.T)) < p).astype(np.float32)

    n_dom = len(cfg.domains[0]) if cfg.domains else 1
    domain_offsets = np.concatenate([[0], np.cumsum(np.bincount(domain, minlength=n_dom))]).astype(np.int64)
    return dict(offsets=offsets.astype(np.int32), indices=indices, lengths=lens,
                dense=dense, labels=labels, mask=mask, domain=domain, domain_offsets=domain_offsets,
                row_base=np.arange(F + 1, dtype=np.int64) * N)


# ---------------------------------------------------------------------------
# parameters
# ---------------------------------------------------------------------------
def _glorot(r, out_f, in_f):
    return r.standard_normal((out_f, in_f)) * math.sqrt(2.0 / (in_f + out_f))


def _mlp(cfg: Config, r, dims):
    layers = []
    for i in range(len(dims) - 1):
        W = _glorot(r, dims[i + 1], dims[i])
        b = r.standard_normal(dims[i + 1]) * 0.01
        layers.append((W, b))
    return layers


def make_dense_params(cfg: Config) -> Dict[str, object]:
    """All non-table parameters as fp32 numpy arrays whose values are exactly
    representable in the storage dtype (weights rounded to bf16 for bf16
    workloads; biases and gains stay fp32)."""
    def w(x):
        return to_storage(x, cfg.dtype).float().numpy()

    def f32(x):
        return np.asarray(x, dtype=np.float32)

    out: Dict[str, object] = {}
    bdims = (cfg.dense_in,) + tuple(cfg.bottom) if cfg.has_dense else ()
    out["bottom"] = [(w(W), f32(b)) for W, b in _mlp(cfg, _rng(cfg.seed, _S_BOTTOM), bdims)] if bdims else []
    tdims = (cfg.top_in,) + tuple(cfg.top)
    out["top"] = [(w(W), f32(b)) for W, b in _mlp(cfg, _rng(cfg.seed, _S_TOP), tdims)]
    if cfg.towers:
        # one tower per objective: objective t's head has weights on its
        # tower's hidden units only, [T, towers]
        T, H = cfg.top[-1], cfg.towers
        assert cfg.top[-2] == T * H, "with towers the last hidden width is T * towers"
        r = _rng(cfg.seed, _S_TOWER)
        out["top"][-1] = (w(_glorot(r, T, H)), f32(r.standard_normal(T) * 0.01))
    if cfg.top_act != "relu":
        # SwishRN gains of the hidden layers: (g_a, g_b) per layer, near 1
        r = _rng(cfg.seed, _S_GAIN)
        out["top_gain"] = [(f32(1.0 + 0.2 * r.standard_normal(o)), f32(1.0 + 0.2 * r.standard_normal(o)))
                           for o in cfg.top[:-1]]
    if cfg.untie:
        # one parameter set per domain for the first `untie` top layers (and
        # their SwishRN gains): W [D, out, in], b [D, out]
        D = len(cfg.domains[0])
        assert cfg.untie <= len(cfg.top) - 1, "untied layers are hidden layers"
        r = _rng(cfg.seed, _S_UNTIE)
        for i in range(cfg.untie):
            o, n = cfg.top[i], tdims[i]
            out["top"][i] = (w(np.stack([_glorot(r, o, n) for _ in range(D)])),
                             f32(r.standard_normal((D, o)) * 0.01))
            if "top_gain" in out:
                out["top_gain"][i] = (f32(1.0 + 0.2 * r.standard_normal((D, o))),
                                      f32(1.0 + 0.2 * r.standard_normal((D, o))))
    n = cfg.n_slots
    if cfg.interact == "fm":
        out["fm_W"] = w(_rng(cfg.seed, _S_FM).standard_normal((n, cfg.fm_rank)) / math.sqrt(n))
    if cfg.interact == "stack":
        layers = []
        r = _rng(cfg.seed, _S_STACK)
        n_l = n
        for l in range(cfg.stack_layers):
            Wl = w(r.standard_normal((n_l, cfg.fm_rank)) / math.sqrt(n_l))
            Al = w(_glorot(r, (cfg.stack_n - cfg.lcb_n) * cfg.d, n_l * cfg.fm_rank))
            Cl = w(_glorot(r, cfg.stack_n, n_l)) if n_l != cfg.stack_n else None
            gl = f32(1.0 + 0.1 * r.standard_normal(cfg.d))
            lay = dict(W=Wl, A=Al, C=Cl, gamma=gl)
            if cfg.lcb_n:
                lay["L"] = w(_glorot(r, cfg.lcb_n, n_l))
            layers.append(lay)
            n_l = cfg.stack_n
        out["stack"] = layers
    return out


def make_tables(cfg: Config, device="cpu", tables: Optional[range] = None) -> torch.Tensor:
    """All embedding tables stacked as one ``[F*rows, d]`` tensor in the
    storage dtype on ``device``.  Table f is drawn from its own torch
    generator, so the same device and seed always give the same values."""
    dt = torch_dtype(cfg.dtype)
    E = torch.empty((cfg.F * cfg.rows, cfg.d), dtype=dt, device=device)
    chunk = max(1, (1 << 26) // cfg.d)
    for f in (tables if tables is not None else range(cfg.F)):
        g = torch.Generator(device=device)
        g.manual_seed(int(cfg.seed) * 4099 + _S_TABLE * 131 + f)
        base = f * cfg.rows
        for r0 in range(0, cfg.rows, chunk):
            r1 = min(cfg.rows, r0 + chunk)
            E[base + r0: base + r1] = (torch.randn((r1 - r0, cfg.d), generator=g, device=device,
                                                   dtype=torch.float32) * 0.01).to(dt)
    return E


# ---------------------------------------------------------------------------
# free-standing operands for per-kernel tests
# ---------------------------------------------------------------------------
def randn(shape, seed: int, stream: int = 0, scale: float = 1.0, dtype: str = "f32") -> np.ndarray:
    """N(0, scale^2) fp32 array, rounded to the storage dtype's values."""
    x = (_rng(seed, _S_AUX + stream).standard_normal(shape) * scale).astype(np.float32)
    if dtype == "bf16":
        x = to_storage(x, "bf16").float().numpy()
    return x


def sub_batch(cfg: Config, batch: Dict[str, np.ndarray], samples):
    """The batch restricted to ``samples`` (all features, feature-major), with
    the table rows it touches renumbered compactly.  Returns
    ``(sub_cfg, sub, global_rows)``: ``global_rows[i]`` is the global table row
    behind compact row ``i``, so the caller gathers the compact table as
    ``E[global_rows]``.  Pure index plumbing."""
    samples = np.asarray(samples, dtype=np.int64)
    B, F = cfg.B, cfg.F
    off = batch["offsets"].astype(np.int64)
    lens, idx_parts, rows_parts, base = [], [], [], [0]
    for f in range(F):
        bags = f * B + samples
        lo, hi = off[bags], off[bags + 1]
        idx = np.concatenate([batch["indices"][a:b] for a, b in zip(lo, hi)]).astype(np.int64) \
            if samples.size else np.zeros(0, np.int64)
        rb = int(batch["row_base"][f])
        uniq, inv = np.unique(idx, return_inverse=True)
        rows_parts.append(rb + uniq)
        idx_parts.append(inv.astype(np.int32))
        lens.append(hi - lo)
        base.append(base[-1] + uniq.size)
    lens = np.concatenate(lens)
    sub = dict(offsets=np.concatenate([[0], np.cumsum(lens)]).astype(np.int32),
               indices=np.concatenate(idx_parts).astype(np.int32),
               row_base=np.array(base, dtype=np.int64),
               dense=batch["dense"][samples], labels=batch["labels"][samples],
               mask=batch["mask"][samples], domain=batch["domain"][samples])
    return cfg.scaled(B=int(samples.size)), sub, np.concatenate(rows_parts)
