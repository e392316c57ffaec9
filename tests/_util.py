"""Shared helpers of the GPU parity tests (test infrastructure)."""
import numpy as np
import torch

import synth
from oracle import mlp as omlp
from oracle import step as ostep
from oracle.metrics import max_rel_err, max_rel_err_normwise

DEV = "cuda"


def tol(cfg):
    """fp32 workloads: 1e-5; bf16-storage workloads: 2e-2 (max relative error)."""
    return 1e-5 if cfg.dtype == "f32" else 2e-2


def assert_close(name, got, ref, t):
    got = got.detach().float().cpu().numpy() if torch.is_tensor(got) else np.asarray(got)
    err = max_rel_err(got, ref)
    print(f"  {name}: max_rel_err={err:.3e} (tol {t:.0e})", flush=True)
    assert err <= t, f"{name}: max_rel_err {err} > {t}"


def assert_close_composed(name, got, ref, t, strict_bound=None):
    """Comparison of a tensor produced by a composed (multi-stage) bf16
    computation: the normwise max relative error must meet t; the element-wise
    row-rms metric must stay under strict_bound (a sanity bound against
    localised bugs; default 3t).  fp32 workloads use the strict metric at t."""
    got = got.detach().float().cpu().numpy() if torch.is_tensor(got) else np.asarray(got)
    strict = max_rel_err(got, ref)
    if t <= 1e-5:
        print(f"  {name}: max_rel_err={strict:.3e} (tol {t:.0e})", flush=True)
        assert strict <= t, f"{name}: max_rel_err {strict} > {t}"
        return
    norm = max_rel_err_normwise(got, ref)
    sb = 3 * t if strict_bound is None else strict_bound
    print(f"  {name}: normwise={norm:.3e} (tol {t:.0e}), element-wise={strict:.3e} (bound {sb:.0e})", flush=True)
    assert norm <= t, f"{name}: normwise max relative error {norm} > {t}"
    assert strict <= sb, f"{name}: element-wise error {strict} > {sb}"


def to_dev(x, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(x))
    if dtype is not None:
        t = t.to(dtype)
    return t.to(DEV)


def stack_dev(layers, sdt):
    """Stack parameters (numpy, from synth) on the device with zeroed gradients."""
    out = []
    for lay in layers:
        def z(x):
            return torch.zeros(x.shape, dtype=torch.float32, device=DEV)
        d = dict(W=to_dev(lay["W"], sdt), A=to_dev(lay["A"], sdt), gamma=to_dev(lay["gamma"]),
                 C=to_dev(lay["C"], sdt) if lay["C"] is not None else None)
        d.update(dW=z(lay["W"]), dA=z(lay["A"]), dgamma=z(lay["gamma"]),
                 dC=z(lay["C"]) if lay["C"] is not None else None)
        out.append(d)
    return out


class Workload:
    """Seeded inputs of a config on the GPU, plus the same values for the oracle."""

    def __init__(self, cfg, batch_id=0, tables=None):
        self.cfg = cfg
        sdt = synth.torch_dtype(cfg.dtype)
        self.batch = synth.make_batch(cfg, batch_id)
        self.params = synth.make_dense_params(cfg)
        self.E = synth.make_tables(cfg, device=DEV) if tables is None else tables
        b = self.batch
        self.offsets = to_dev(b["offsets"])
        self.indices = to_dev(b["indices"])
        self.row_base = to_dev(b["row_base"])
        self.dense = to_dev(b["dense"], sdt)
        self.labels = to_dev(b["labels"])
        self.mask = to_dev(b["mask"])
        self.nnz = int(b["offsets"][-1])

        def lin(W, bb):
            return dict(W=to_dev(W, sdt), b=to_dev(bb),
                        dW=torch.zeros(W.shape, dtype=torch.float32, device=DEV),
                        db=torch.zeros(bb.shape, dtype=torch.float32, device=DEV))

        self.bottom = [lin(W, bb) for W, bb in self.params["bottom"]]
        self.top = [lin(W, bb) for W, bb in self.params["top"]]
        self.fm_W = to_dev(self.params["fm_W"], sdt) if "fm_W" in self.params else None
        self.fm_dW = torch.zeros(self.fm_W.shape, dtype=torch.float32, device=DEV) \
            if self.fm_W is not None else None
        self.stack = stack_dev(self.params["stack"], sdt) if "stack" in self.params else None

    def table_np(self):
        return self.E.float().cpu().double().numpy()

    def step_model(self):
        from paper_2512_09200_amd import api
        c = self.cfg
        return api.StepModel(tables=self.E, row_base=self.row_base, num_features=c.F,
                             dense_in=c.dense_in, bottom=self.bottom, top=self.top,
                             interact=c.interact, fm_W=self.fm_W, fm_dW=self.fm_dW, pool=c.pool,
                             stack=self.stack, stack_n=c.stack_n, ln_eps=c.ln_eps)


def relu_overrides(cfg, params, table, batch, gpu_in, gpu_out, max_iter=4):
    """ReLU decisions that the GPU may legitimately take the other way.

    A decision is ambiguous when the float64 pre-activation ``a`` lies within
    ``band = fp32 accumulation bound + |h_gpu - h_ref| @ |W|^T`` of zero: the
    first term covers summation order in fp32, the second the observed
    differences of the layer's (bf16-stored) inputs, which are themselves
    checked against the oracle by the caller.  There the GPU's decision is
    accepted after checking its value is consistent with a pre-activation that
    small; everywhere else the oracle decides.  Iterates until the set is
    stable.  gpu_in / gpu_out: dict "bottom"/"top" -> per-layer input / output
    tensors (None where absent).  Returns (overrides, n_band, n_flipped)."""
    overrides = None
    for _ in range(max_iter):
        c = ostep.forward(cfg, params, table, batch, overrides)
        new, n_band, n_flip = {}, 0, 0
        for name, hs_key, mk, layers in (("bottom", "hs_bottom", "masks_bottom", params["bottom"]),
                                          ("top", "hs_top", "masks_top", params["top"])):
            if hs_key not in c:
                continue
            hs = c[hs_key]
            ov = []
            for i, (W, b) in enumerate(layers):
                out_t = gpu_out[name][i] if i < len(gpu_out[name]) else None
                in_t = gpu_in[name][i] if i < len(gpu_in[name]) else None
                if out_t is None or c[mk][i] is None:
                    ov.append(None)
                    continue
                h_ref = hs[i]
                a = omlp.linear(h_ref, W, b)
                band = omlp.relu_band(h_ref, W, b)
                if in_t is not None:
                    h_gpu = in_t.float().cpu().double().numpy()
                    band = band + np.abs(h_gpu - h_ref) @ np.abs(np.asarray(W, np.float64)).T
                where = np.abs(a) <= band
                g = out_t.float().cpu().double().numpy()
                assert np.all(np.abs(g[where]) <= 2.01 * band[where] + 1e-30), f"{name}{i}: GPU value outside band"
                pos = g > 0
                n_band += int(where.sum())
                n_flip += int((where & (pos != (a > 0))).sum())
                ov.append((where, pos))
            new[name] = ov
        same = overrides is not None and all(
            (x is None and y is None) or (x is not None and y is not None and np.array_equal(x[0], y[0])
                                          and np.array_equal(x[1], y[1]))
            for k in new for x, y in zip(new[k], overrides[k]))
        overrides = new
        if same:
            break
    return overrides, n_band, n_flip
