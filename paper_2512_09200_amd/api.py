"""Torch-facing binding of the C ABI: the same entry-point names as
include/lattice.h, taking torch tensors that live on the GPU.  Argument
marshalling and buffer allocation only -- every step runs in liblattice.so.
"""
import ctypes
from ctypes import byref

import torch

from . import _abi as A
from ._abi import check, load

_POOL = {"sum": A.POOL_SUM, "mean": A.POOL_MEAN}
_KIND = {"dot": A.DOT, "fm": A.FM, "stack": A.STACK}


def _p(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _dt(t):
    if t.dtype == torch.bfloat16:
        return A.BF16
    if t.dtype == torch.float32:
        return A.F32
    raise TypeError(f"unsupported dtype {t.dtype}")


def _stream(stream):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _row_stride(t):
    if t.dim() != 2:
        raise ValueError("expected a 2-D tensor")
    if t.shape[0] == 0:
        return t.shape[1]            # no rows: any stride >= the width
    if t.stride(1) != 1 and t.shape[1] > 1:
        raise ValueError("expected a 2-D tensor with unit column stride")
    return t.stride(0)


def _contig(*ts):
    for t in ts:
        if t is not None and not t.is_contiguous():
            raise ValueError("tensor must be contiguous")


def table_max_rows(row_base):
    """Rows of the largest table (one device-to-host copy of row_base)."""
    rb = row_base.cpu()
    return int((rb[1:] - rb[:-1]).max()) if rb.numel() > 1 else 0


def _tables(table, row_base, max_rows=None):
    """max_rows None: derived from row_base (a synchronising copy); 0: unknown."""
    _contig(table, row_base)
    if max_rows is None:
        max_rows = table_max_rows(row_base)
    return A.lattice_tables(data=table.data_ptr(), dtype=_dt(table), dim=table.shape[1],
                            total_rows=table.shape[0], row_base=row_base.data_ptr(),
                            max_rows=int(max_rows))


def _jagged(offsets, indices, F, B):
    _contig(offsets, indices)
    return A.lattice_jagged(num_features=F, batch=B, offsets=offsets.data_ptr(),
                            indices=indices.data_ptr() if indices.numel() else None,
                            nnz=indices.numel())


# ---------------------------------------------------------------------------
def lattice_embbag_fwd(table, row_base, offsets, indices, F, B, X, first_slot=0, pool="sum",
                       stream=None):
    _contig(X)
    lib = load()
    t, j = _tables(table, row_base, 0), _jagged(offsets, indices, F, B)
    check(lib.lattice_embbag_fwd(byref(t), byref(j), _POOL[pool], _p(X), _dt(X), X.shape[1],
                                 first_slot, _stream(stream)))
    return X


def lattice_embbag_bwd_noalloc(table, row_base, offsets, indices, F, B, dX, out, first_slot=0, lr=0.0,
                               pool="sum", stream=None, max_rows=None):
    """lattice_embbag_bwd without a workspace (the library's own per-GPU
    scratch array); out: dict of preallocated output tensors as returned by
    lattice_embbag_bwd (unique_rows, seg_offsets, sorted_bags, num_unique,
    grad_rows or None).  Allocates nothing."""
    _contig(dX)
    lib = load()
    t, j = _tables(table, row_base, max_rows), _jagged(offsets, indices, F, B)
    sg = A.lattice_sparse_grad(*(o.data_ptr() if o is not None else None for o in
                                 (out["unique_rows"], out["seg_offsets"], out["sorted_bags"],
                                  out["num_unique"], out.get("grad_rows"))))
    check(lib.lattice_embbag_bwd_noalloc(byref(t), byref(j), _POOL[pool], _p(dX), _dt(dX), dX.shape[1],
                                         first_slot, byref(sg), float(lr), _stream(stream)))
    return out


def lattice_embbag_bwd(table, row_base, offsets, indices, F, B, dX, first_slot=0, lr=0.0,
                       pool="sum", emit_grad_rows=True, stream=None, max_rows=None):
    """Returns dict(unique_rows, seg_offsets, sorted_bags, num_unique, grad_rows); with lr != 0
    the table is updated in place.  max_rows: rows of the largest table (None: from row_base)."""
    _contig(dX)
    lib = load()
    t, j = _tables(table, row_base, max_rows), _jagged(offsets, indices, F, B)
    nnz = indices.numel()
    dev = table.device
    n = max(nnz, 1)
    out = dict(unique_rows=torch.empty(n, dtype=torch.int32, device=dev),
               seg_offsets=torch.empty(n + 1, dtype=torch.int32, device=dev),
               sorted_bags=torch.empty(n, dtype=torch.int32, device=dev),
               num_unique=torch.empty(1, dtype=torch.int32, device=dev),
               grad_rows=torch.empty((n, table.shape[1]), dtype=torch.float32, device=dev)
               if emit_grad_rows else None)
    sg = A.lattice_sparse_grad(*(o.data_ptr() if o is not None else None for o in
                                 (out["unique_rows"], out["seg_offsets"], out["sorted_bags"],
                                  out["num_unique"], out["grad_rows"])))
    wsb = lib.lattice_embbag_bwd_workspace(byref(t), byref(j))
    ws = torch.empty(max(wsb, 1), dtype=torch.uint8, device=dev)
    check(lib.lattice_embbag_bwd(byref(t), byref(j), _POOL[pool], _p(dX), _dt(dX), dX.shape[1],
                                 first_slot, byref(sg), float(lr), _p(ws), wsb, _stream(stream)))
    return out


def lattice_validate_batch(table, row_base, offsets, indices, F, B, stream=None, max_rows=None):
    """Returns (ok, first_bad)."""
    lib = load()
    t, j = _tables(table, row_base, max_rows), _jagged(offsets, indices, F, B)
    bad = ctypes.c_int64(0)
    st = lib.lattice_validate_batch(byref(t), byref(j), byref(bad), _stream(stream))
    if st == 4:
        return False, bad.value
    check(st)
    return True, 0


# ---------------------------------------------------------------------------
def _ptr(t):
    return t.data_ptr() if t is not None else None


def stack_layers(layers):
    """layers: list of dicts W, A, C (or None), gamma, dW, dA, dC, dgamma, and
    for full fusion blocks L, dL (device tensors)."""
    arr = (A.lattice_stack_layer * len(layers))()
    for i, L in enumerate(layers):
        _contig(*(L.get(k) for k in ("W", "A", "C", "gamma", "L")))
        arr[i] = A.lattice_stack_layer(*(_ptr(L.get(k)) for k in
                                         ("W", "A", "C", "gamma", "dW", "dA", "dC", "dgamma", "L", "dL")))
    return arr


def _lcb_n(stack):
    return int(stack[0]["L"].shape[0]) if stack and stack[0].get("L") is not None else 0


def interact_desc(kind, X, emit_slot0, fm_W=None, fm_dW=None, rank=0, stack=None, stack_n=0,
                  ln_eps=1e-5, slot_mask=None, fp8_proj=None):
    """stack: list of layer dicts (see stack_layers) for kind "stack";
    slot_mask (DOT): int32 [B, 4] device tensor of per-sample slot bits;
    fp8_proj (STACK): None, "precise" or "fast" (the FM projection in FP8)."""
    arr = stack_layers(stack) if stack else None
    if stack:
        rank = stack[0]["W"].shape[1]
    d = A.lattice_interact_desc(kind=_KIND[kind], dtype=_dt(X), n=X.shape[1], dim=X.shape[2],
                                rank=(fm_W.shape[1] if fm_W is not None else rank),
                                emit_slot0=int(emit_slot0), fm_W=_ptr(fm_W), fm_dW=_ptr(fm_dW),
                                n_layers=len(stack) if stack else 0, stack_n=stack_n,
                                ln_eps=ln_eps, layers=arr, lcb_n=_lcb_n(stack),
                                slot_mask=_ptr(slot_mask), fp8_proj=_FP8_TOP[fp8_proj])
    d._keep = arr
    return d


def lattice_interact_fwd(kind, X, out, emit_slot0=False, fm_W=None, stream=None, stack=None,
                         stack_n=0, ln_eps=1e-5, slot_mask=None, fp8_proj=None):
    """Returns the workspace (saved state), which lattice_interact_bwd needs."""
    _contig(X, fm_W, slot_mask)
    lib = load()
    d = interact_desc(kind, X, emit_slot0, fm_W, stack=stack, stack_n=stack_n, ln_eps=ln_eps,
                      slot_mask=slot_mask, fp8_proj=fp8_proj)
    wsb = lib.lattice_interact_workspace(byref(d), X.shape[0])
    ws = torch.empty(max(wsb, 1), dtype=torch.uint8, device=X.device)
    check(lib.lattice_interact_fwd(byref(d), X.shape[0], _p(X), _p(out), _row_stride(out), _p(ws),
                                   wsb, _stream(stream)))
    return ws


def lattice_interact_bwd(kind, X, d_out, dX, emit_slot0=False, fm_W=None, fm_dW=None, stream=None,
                         stack=None, stack_n=0, ln_eps=1e-5, ws=None, slot_mask=None, fp8_proj=None):
    _contig(X, dX, fm_W, fm_dW, slot_mask)
    lib = load()
    d = interact_desc(kind, X, emit_slot0, fm_W, fm_dW, stack=stack, stack_n=stack_n, ln_eps=ln_eps,
                      slot_mask=slot_mask, fp8_proj=fp8_proj)
    wsb = lib.lattice_interact_workspace(byref(d), X.shape[0])
    if ws is None:
        ws = torch.empty(max(wsb, 1), dtype=torch.uint8, device=X.device)
    check(lib.lattice_interact_bwd(byref(d), X.shape[0], _p(X), _p(d_out), _row_stride(d_out),
                                   _p(dX), _p(ws), ws.numel(), _stream(stream)))
    return dX


# ---------------------------------------------------------------------------
_ACT = {None: A.ACT_RELU, "relu": A.ACT_RELU, "swishrn": A.ACT_SWISHRN, "hardswishrn": A.ACT_HARDSWISHRN}


def mlp_desc(layers, relu_last, dtype, act=None, norm_block=A.BLOCKNORM_COLS, norm_eps=1e-6,
             tower_heads=False, n_domains=0, untied_layers=0, domain_offsets=None):
    """layers: list of dicts with W, b (optional), dW, db (optional); SwishRN
    layers (act "swishrn" / "hardswishrn") also gain [2, out] fp32, dgain
    (optional), and for lattice_mlp_heads_fwd/bwd pre [B, out] (storage
    dtype) and rinv [B, groups] fp32.  Untied layers (the first
    untied_layers, n_domains >= 2) hold stacked sets: W [D, out, in],
    b [D, out], gain [D, 2, out] and gradients alike; domain_offsets (host,
    [D + 1]) groups the rows for lattice_mlp_heads_fwd/bwd."""
    arr = (A.lattice_linear * len(layers))()
    for i, L in enumerate(layers):
        W = L["W"]
        _contig(W)
        # tower heads: W is [T, H] and the layer's input holds T groups of H;
        # untied layers: W is [D, out, in]
        in_dim = W.shape[0] * W.shape[1] if (tower_heads and i == len(layers) - 1) else W.shape[-1]
        arr[i] = A.lattice_linear(in_dim=in_dim, out_dim=W.shape[-2], W=W.data_ptr(),
                                  b=_ptr(L.get("b")), dW=_ptr(L.get("dW")), db=_ptr(L.get("db")),
                                  gain=_ptr(L.get("gain")), dgain=_ptr(L.get("dgain")),
                                  pre=_ptr(L.get("pre")), rinv=_ptr(L.get("rinv")))
    d = A.lattice_mlp_desc(dtype=dtype, n_layers=len(layers), layers=arr, relu_last=int(relu_last),
                           act=_ACT[act], norm_block=int(norm_block), norm_eps=float(norm_eps),
                           tower_heads=int(bool(tower_heads)), n_domains=int(n_domains),
                           untied_layers=int(untied_layers))
    d._keep = [arr]
    if domain_offsets is not None:
        off = (ctypes.c_int64 * len(domain_offsets))(*[int(x) for x in domain_offsets])
        d.domain_offsets = ctypes.cast(off, ctypes.POINTER(ctypes.c_int64))
        d._keep.append(off)
    return d


def swishrn_groups(N, norm_block):
    """Normalisation groups of a SwishRN layer of width N (columns of rinv)."""
    return 1 if norm_block <= 0 or norm_block >= N else -(-N // norm_block)


def lattice_mlp_heads_fwd(layers, x, acts, relu_last, loss=None, stream=None, act=None,
                          norm_block=A.BLOCKNORM_COLS, norm_eps=1e-6, tower_heads=False, n_domains=0,
                          untied_layers=0, domain_offsets=None):
    """acts: list of output tensors (2-D, unit column stride); loss: optional
    dict(labels, mask, loss, d_logits, d_logits_op); act / norm_block /
    norm_eps: the activation, tower_heads: the last layer is the heads of
    per-objective towers; n_domains / untied_layers / domain_offsets:
    parameter untying (see mlp_desc)."""
    lib = load()
    d = mlp_desc(layers, relu_last, _dt(x), act, norm_block, norm_eps, tower_heads, n_domains, untied_layers,
                 domain_offsets)
    n = len(layers)
    ptrs = (ctypes.c_void_p * n)(*[a.data_ptr() for a in acts])
    strides = (ctypes.c_int64 * n)(*[_row_stride(a) for a in acts])
    ld = None
    if loss is not None:
        ld = A.lattice_loss_desc(labels=loss["labels"].data_ptr(), mask=loss["mask"].data_ptr(),
                                 loss=loss["loss"].data_ptr(), d_logits=loss["d_logits"].data_ptr(),
                                 d_logits_op=loss["d_logits_op"].data_ptr()
                                 if loss.get("d_logits_op") is not None else None)
    wsb = lib.lattice_mlp_heads_workspace(byref(d), x.shape[0])
    ws = torch.empty(max(wsb, 1), dtype=torch.uint8, device=x.device)
    check(lib.lattice_mlp_heads_fwd(byref(d), x.shape[0], _p(x), _row_stride(x), ptrs, strides,
                                    byref(ld) if ld is not None else None, _p(ws), wsb,
                                    _stream(stream)))


def lattice_mlp_heads_bwd(layers, x, acts, d_out, relu_last, d_in=None, stream=None, act=None,
                          norm_block=A.BLOCKNORM_COLS, norm_eps=1e-6, tower_heads=False, n_domains=0,
                          untied_layers=0, domain_offsets=None):
    lib = load()
    d = mlp_desc(layers, relu_last, _dt(x), act, norm_block, norm_eps, tower_heads, n_domains, untied_layers,
                 domain_offsets)
    n = len(layers)
    ptrs = (ctypes.c_void_p * n)(*[a.data_ptr() for a in acts])
    strides = (ctypes.c_int64 * n)(*[_row_stride(a) for a in acts])
    wsb = lib.lattice_mlp_heads_workspace(byref(d), x.shape[0])
    ws = torch.empty(max(wsb, 1), dtype=torch.uint8, device=x.device)
    check(lib.lattice_mlp_heads_bwd(byref(d), x.shape[0], _p(x), _row_stride(x), ptrs, strides,
                                    _p(d_out), _row_stride(d_out), _p(d_in),
                                    _row_stride(d_in) if d_in is not None else 0, _p(ws), wsb,
                                    _stream(stream)))


# ---------------------------------------------------------------------------
_FP8_SCALING = {"row": A.FP8_ROWWISE, "tensor": A.FP8_TENSORWISE}


def fp8_ld(cols):
    """Row stride (bytes) of the e4m3 codes of a matrix with `cols` columns."""
    return (cols + 15) // 16 * 16


def lattice_fp8_quantize(x, scaling="row", stream=None):
    """e4m3 codes [rows, fp8_ld(cols)] (uint8) and fp32 scales ([rows] or [1])
    of a 2-D bf16 / fp32 tensor (unit column stride)."""
    lib = load()
    rows, cols = x.shape
    q = torch.empty((rows, fp8_ld(cols)), dtype=torch.uint8, device=x.device)
    sc = torch.empty((rows if scaling == "row" else 1,), dtype=torch.float32, device=x.device)
    wsb = lib.lattice_fp8_quantize_workspace()
    ws = torch.empty(wsb, dtype=torch.uint8, device=x.device)
    check(lib.lattice_fp8_quantize(_p(x), _dt(x), rows, cols, _row_stride(x), _FP8_SCALING[scaling], _p(q),
                                   q.stride(0), _p(sc), _p(ws), wsb, _stream(stream)))
    return q, sc


def lattice_linear_fp8_fwd(qa, sa, qw, sw, K, bias=None, relu=False, out=None, out_dtype=torch.bfloat16,
                           fast_accum=False, stream=None):
    """Y = act(deq(qa) deq(qw)^T + bias) from e4m3 codes and their scales
    (row-wise when the scale vector has one entry per row); fast_accum as in
    lattice.h (False: per-64-k partial sums added in fp32)."""
    lib = load()
    M, N = qa.shape[0], qw.shape[0]
    if out is None:
        out = torch.empty((M, N), dtype=out_dtype, device=qa.device)
    a_sc = A.FP8_ROWWISE if sa.numel() == M and M > 1 else A.FP8_TENSORWISE
    w_sc = A.FP8_ROWWISE if sw.numel() == N and N > 1 else A.FP8_TENSORWISE
    check(lib.lattice_linear_fp8_fwd(_p(qa), qa.stride(0), _p(sa), a_sc, _p(qw), qw.stride(0), _p(sw), w_sc,
                                     _p(bias), M, N, K, int(bool(relu)), int(bool(fast_accum)), _p(out), _dt(out),
                                     _row_stride(out), _stream(stream)))
    return out


# ---------------------------------------------------------------------------
class StepModel:
    """Marshals a model's device tensors into a lattice_model_desc.

    tables [R, d], row_base int64 [F+1]; bottom/top: lists of dicts
    {W, b, dW, db} (SwishRN top layers: also gain, dgain); fm_W / fm_dW for
    the FM interaction; max_rows: rows of the largest table (None: read from
    row_base once, here); top_act: None / "relu", "swishrn" or "hardswishrn"
    for the top MLP's hidden layers; towers: the top MLP's last layer is the
    heads of per-objective towers (its W [T, H]); n_domains / untied_layers:
    the first untied_layers top layers hold one parameter set per domain
    (lattice_step then takes the batch's domain_offsets); skip_absent
    (DOT): whole features may be absent from a sample (empty bags), so the
    step's DOT forward skips the empty slots; fp8_proj (STACK): None,
    "precise" or "fast" -- the FM projection in FP8."""

    def __init__(self, *, tables, row_base, num_features, dense_in, bottom, top, interact,
                 fm_W=None, fm_dW=None, pool="sum", stack=None, stack_n=0, ln_eps=1e-5,
                 max_rows=None, top_act=None, norm_block=A.BLOCKNORM_COLS, norm_eps=1e-6,
                 towers=False, n_domains=0, untied_layers=0, skip_absent=False, fp8_proj=None):
        _contig(tables, row_base)
        dt = _dt(tables)
        d = tables.shape[1]
        n = num_features + (1 if dense_in > 0 else 0)
        self._bottom = mlp_desc(bottom, True, dt) if dense_in > 0 else A.lattice_mlp_desc(dtype=dt)
        self._top = mlp_desc(top, False, dt, top_act, norm_block, norm_eps, tower_heads=towers,
                             n_domains=n_domains, untied_layers=untied_layers)
        self.top_act, self.norm_block = top_act, norm_block
        self._stack = stack_layers(stack) if stack else None
        rank = fm_W.shape[1] if fm_W is not None else (stack[0]["W"].shape[1] if stack else 0)
        idesc = A.lattice_interact_desc(kind=_KIND[interact], dtype=dt, n=n, dim=d, rank=rank,
                                        emit_slot0=int(dense_in > 0 and interact != "stack"),
                                        fm_W=_ptr(fm_W), fm_dW=_ptr(fm_dW),
                                        n_layers=len(stack) if stack else 0, stack_n=stack_n,
                                        ln_eps=ln_eps, layers=self._stack, lcb_n=_lcb_n(stack),
                                        skip_absent=int(bool(skip_absent)),
                                        fp8_proj=_FP8_TOP[fp8_proj])
        self.desc = A.lattice_model_desc(dtype=dt, pool=_POOL[pool],
                                         tables=_tables(tables, row_base, max_rows),
                                         num_features=num_features, dense_in=dense_in,
                                         bottom=self._bottom, interact=idesc, top=self._top)
        self.tensors = dict(tables=tables, row_base=row_base, bottom=bottom, top=top, fm_W=fm_W,
                            fm_dW=fm_dW, stack=stack)
        self.device = tables.device
        self.num_features = num_features
        self.dense_in = dense_in
        self.n = n
        self.d = d


_FP8_TOP = {None: 0, False: 0, "precise": 1, "fast": 2}


def lattice_step_plan(model, B, nnz, lr_tables=0.0, emit_grad_rows=False, fp8_top=None):
    """Layout of a workspace for batches of B samples and up to nnz lookups;
    pass the same nnz as nnz_capacity (and the same fp8_top) to lattice_step."""
    lib = load()
    opts = A.lattice_step_opts(lr_tables=float(lr_tables), emit_grad_rows=int(emit_grad_rows),
                               nnz_capacity=int(nnz), fp8_top=_FP8_TOP[fp8_top])
    lay = A.lattice_step_layout()
    check(lib.lattice_step_plan(byref(model.desc), B, nnz, byref(opts), byref(lay)))
    return lay


class SideStream:
    """A second stream of the caller's device and the fork / join events that
    lattice_step uses to overlap the bottom MLP and the sparse gradient's
    sort with the rest of the step (default priority; the
    events are created here, by torch, and recorded once so they exist)."""

    def __init__(self, device=None):
        self.stream = torch.cuda.Stream(device=device)
        self.events = [torch.cuda.Event() for _ in range(A.SIDE_EVENTS)]
        for e in self.events:
            e.record(self.stream)
        self._arr = (ctypes.c_void_p * A.SIDE_EVENTS)(*[e.cuda_event for e in self.events])

    def ptrs(self):
        return self.stream.cuda_stream, ctypes.cast(self._arr, ctypes.POINTER(ctypes.c_void_p))


def lattice_step(model, offsets, indices, dense, labels, mask, ws, lr_tables=0.0,
                 emit_grad_rows=False, stream=None, stage_events=None, nnz_capacity=0,
                 side=None, fp8_top=None, domain_offsets=None):
    """One forward+backward step; ws is a uint8 device tensor of at least
    lattice_step_plan(...).total_bytes.  stage_events: optional list of
    2*len(STAGES) torch.cuda.Event(enable_timing=True) or None: [2s] and
    [2s+1] are recorded when stage s begins and ends, on the stream that runs
    it (None: not recorded).
    side: a SideStream to overlap the bottom MLP and the sort on (None:
    every stage on the step's stream).  fp8_top: None, "precise" or "fast"
    (the top MLP's hidden-layer forward in FP8; see lattice.h).
    domain_offsets: host [D + 1] offsets of the domain-grouped samples
    (models with untied layers)."""
    lib = load()
    _contig(dense, labels, mask, ws)
    B = labels.shape[0]
    batch = A.lattice_batch_desc(bags=_jagged(offsets, indices, model.num_features, B),
                                 dense=dense.data_ptr() if dense is not None and dense.numel() else None,
                                 labels=labels.data_ptr(), mask=mask.data_ptr())
    if domain_offsets is not None:       # host offsets of the domain-grouped samples
        off = (ctypes.c_int64 * len(domain_offsets))(*[int(x) for x in domain_offsets])
        batch.domain_offsets = ctypes.cast(off, ctypes.POINTER(ctypes.c_int64))
    opts = A.lattice_step_opts(lr_tables=float(lr_tables), emit_grad_rows=int(emit_grad_rows),
                               nnz_capacity=int(nnz_capacity or indices.numel()), fp8_top=_FP8_TOP[fp8_top])
    if side is not None:
        opts.side_stream, opts.side_events = side.ptrs()
    if stage_events is not None:
        if len(stage_events) != 2 * len(A.STAGES):
            raise ValueError("need 2*len(STAGES) events")
        arr = (ctypes.c_void_p * len(stage_events))(*[e.cuda_event if e is not None else None
                                                       for e in stage_events])
        opts.stage_events = ctypes.cast(arr, ctypes.POINTER(ctypes.c_void_p))
    check(lib.lattice_step(byref(model.desc), byref(batch), byref(opts), _p(ws), ws.numel(),
                           _stream(stream)))


def lattice_forward(model, offsets, indices, dense, B, ws, stream=None, nnz_capacity=0, side=None,
                    fp8_top=None, domain_offsets=None):
    """The step's forward alone (inference): logits at layout.logits of ws
    (see step_views); no labels, gradients or table update.  The same plan
    and workspace as lattice_step."""
    lib = load()
    _contig(dense, ws)
    batch = A.lattice_batch_desc(bags=_jagged(offsets, indices, model.num_features, B),
                                 dense=dense.data_ptr() if dense is not None and dense.numel() else None)
    if domain_offsets is not None:
        off = (ctypes.c_int64 * len(domain_offsets))(*[int(x) for x in domain_offsets])
        batch.domain_offsets = ctypes.cast(off, ctypes.POINTER(ctypes.c_int64))
    opts = A.lattice_step_opts(nnz_capacity=int(nnz_capacity or indices.numel()), fp8_top=_FP8_TOP[fp8_top])
    if side is not None:
        opts.side_stream, opts.side_events = side.ptrs()
    check(lib.lattice_forward(byref(model.desc), byref(batch), byref(opts), _p(ws), ws.numel(),
                              _stream(stream)))


def step_views(model, ws, layout, B, T, nnz):
    """Torch views of the step's intermediates inside the workspace."""
    dt = model.tensors["tables"].dtype
    es = 2 if dt == torch.bfloat16 else 4

    def view(off, shape, dtype):
        if off < 0:
            return None
        n = 1
        for s in shape:
            n *= s
        size = n * torch.empty((), dtype=dtype).element_size()
        return ws[off: off + size].view(dtype).view(*shape)

    n, d = model.n, model.d
    v = dict(X=view(layout.X, (B, n, d), dt), t=view(layout.t, (B, layout.t_stride), dt),
             logits=view(layout.logits, (B, T), torch.float32),
             d_logits=view(layout.d_logits, (B, T), torch.float32),
             loss=view(layout.loss, (1,), torch.float32),
             d_t=view(layout.d_t, (B, layout.t_stride), dt), dX=view(layout.dX, (B, n, d), dt),
             unique_rows=view(layout.unique_rows, (max(nnz, 1),), torch.int32),
             seg_offsets=view(layout.seg_offsets, (max(nnz, 1) + 1,), torch.int32),
             sorted_bags=view(layout.sorted_bags, (max(nnz, 1),), torch.int32),
             num_unique=view(layout.num_unique, (1,), torch.int32),
             grad_rows=view(layout.grad_rows, (max(nnz, 1), d), torch.float32))
    tops = model.tensors["top"]
    v["top_act"] = [view(layout.top_act[i], (B, tops[i]["W"].shape[-2]), dt) for i in range(len(tops) - 1)]
    v["top_grad"] = [view(layout.top_grad[i], (B, tops[i]["W"].shape[-2]), dt) for i in range(len(tops))]
    outs = [tops[i]["W"].shape[-2] for i in range(len(tops) - 1)]
    v["top_pre"] = [view(layout.top_pre[i], (B, o), dt) for i, o in enumerate(outs)]
    v["top_rinv"] = [view(layout.top_rinv[i], (B, swishrn_groups(o, model.norm_block)), torch.float32)
                     for i, o in enumerate(outs)]
    v["top_gout"] = [view(layout.top_gout[i], (B, o), dt) for i, o in enumerate(outs)]
    bots = model.tensors["bottom"]
    v["bottom_act"] = [view(layout.bottom_act[i], (B, bots[i]["W"].shape[0]), dt)
                       for i in range(len(bots) - 1)] if model.dense_in > 0 else []
    v["bottom_grad"] = [view(layout.bottom_grad[i], (B, bots[i]["W"].shape[0]), dt)
                        for i in range(len(bots))] if model.dense_in > 0 else []
    _ = es
    # the stacked interaction's saved state (per layer P, F, H, mean, rstd, X_{l+1})
    v["stack_state"] = None
    if model.desc.interact.kind == _KIND["stack"]:
        st = stack_state_offsets(model.desc.interact, B)
        base = layout.interact
        nl, nv, k = model.desc.interact.n_layers, model.desc.interact.stack_n, model.desc.interact.rank
        layers = []
        for l in range(nl):
            nin = n if l == 0 else nv
            layers.append(dict(
                P=view(base + st.P[l], (B, d, k), dt), F=view(base + st.F[l], (B, nin, k), dt),
                H=view(base + st.H[l], (B, nv * d), torch.float32),
                mean=view(base + st.mean[l], (B, nv), torch.float32),
                rstd=view(base + st.rstd[l], (B, nv), torch.float32),
                Xn=view(base + st.Xn[l], (B, nv, d), dt) if st.Xn[l] >= 0 else None))
        v["stack_state"] = layers
    return v


def stack_state_offsets(idesc, B):
    """lattice_stack_state of an interaction descriptor (byte offsets of the
    saved state inside its workspace)."""
    out = A.lattice_stack_state()
    check(load().lattice_interact_state(byref(idesc), B, byref(out)))
    return out


def lattice_interact_state(kind, X, stack, stack_n, ws, ln_eps=1e-5, fp8_proj=None):
    """Views of the stacked interaction's saved state inside ws (the workspace
    lattice_interact_fwd returned): per layer P, F, H, mean, rstd, X_{l+1}."""
    d_ = interact_desc(kind, X, False, stack=stack, stack_n=stack_n, ln_eps=ln_eps, fp8_proj=fp8_proj)
    st = stack_state_offsets(d_, X.shape[0])
    B, n, dd = X.shape
    k = stack[0]["W"].shape[1]

    def view(off, shape, dtype):
        size = 1
        for x in shape:
            size *= int(x)
        size *= torch.empty((), dtype=dtype).element_size()
        return ws[off: off + size].view(dtype).view(*shape)
    out = []
    for l in range(len(stack)):
        nin = n if l == 0 else stack_n
        out.append(dict(P=view(st.P[l], (B, dd, k), X.dtype), F=view(st.F[l], (B, nin, k), X.dtype),
                        H=view(st.H[l], (B, stack_n * dd), torch.float32),
                        mean=view(st.mean[l], (B, stack_n), torch.float32),
                        rstd=view(st.rstd[l], (B, stack_n), torch.float32),
                        Xn=view(st.Xn[l], (B, stack_n, dd), X.dtype) if st.Xn[l] >= 0 else None))
    return out
