"""Every error status that include/lattice.h promises, hit through the C ABI
on a machine without a GPU: all of them are raised by argument checks that
run before anything is enqueued, so no device memory is touched (the
non-null pointers below are placeholders that are never dereferenced).  The
valid no-op cases that write nothing (forward calls with B = 0 or F*B = 0)
return LATTICE_OK the same way."""
import ctypes
from ctypes import byref

import pytest

from paper_2512_09200_amd import _abi as A

OK, INVALID_ARG, UNSUPPORTED, WORKSPACE = 0, 1, 2, 3
FAKE = 0x10000          # placeholder device pointer, never dereferenced here


def _gpu_visible():
    try:
        import torch
        return torch.cuda.device_count() > 0
    except Exception:
        return False


# A check that unexpectedly passed would enqueue work on placeholder
# pointers: these tests only ever run where no GPU is visible.
pytestmark = pytest.mark.skipif(_gpu_visible(), reason="placeholder pointers must never reach a GPU")


@pytest.fixture(scope="module")
def lib():
    return A.load()


def last_error(lib):
    return lib.lattice_last_error().decode()


def tables(dim=128, dtype=A.BF16, total_rows=1000, max_rows=0, data=FAKE):
    return A.lattice_tables(data=data, dtype=dtype, dim=dim, total_rows=total_rows,
                            row_base=FAKE, max_rows=max_rows)


def bags(F=2, B=4, nnz=10):
    return A.lattice_jagged(num_features=F, batch=B, offsets=FAKE, indices=FAKE, nnz=nnz)


# ------------------------------------------------------------- pooled lookup
def test_embbag_fwd_statuses(lib):
    t, j = tables(), bags()
    f = lib.lattice_embbag_fwd
    assert f(None, byref(j), A.POOL_SUM, FAKE, A.BF16, 3, 1, None) == INVALID_ARG
    assert "null" in last_error(lib)
    assert f(byref(t), None, A.POOL_SUM, FAKE, A.BF16, 3, 1, None) == INVALID_ARG
    assert f(byref(tables(data=None)), byref(j), A.POOL_SUM, FAKE, A.BF16, 3, 1, None) == INVALID_ARG
    for dim in (12, 0, 264, -8):
        assert f(byref(tables(dim=dim)), byref(j), A.POOL_SUM, FAKE, A.BF16, 3, 1, None) == UNSUPPORTED, dim
        assert "dim" in last_error(lib)
    # first_slot + F > n_slots
    assert f(byref(t), byref(j), A.POOL_SUM, FAKE, A.BF16, 2, 1, None) == INVALID_ARG
    assert "slots" in last_error(lib)
    assert f(byref(t), byref(j), 7, FAKE, A.BF16, 3, 1, None) == INVALID_ARG       # pool mode
    assert f(byref(t), byref(j), A.POOL_SUM, FAKE, 9, 3, 1, None) == INVALID_ARG   # X dtype
    assert f(byref(t), byref(bags(nnz=-1)), A.POOL_SUM, FAKE, A.BF16, 3, 1, None) == INVALID_ARG
    assert f(byref(t), byref(bags(nnz=1 << 31)), A.POOL_SUM, FAKE, A.BF16, 3, 1, None) == INVALID_ARG
    assert f(byref(tables(total_rows=1 << 31)), byref(j), A.POOL_SUM, FAKE, A.BF16, 3, 1, None) == UNSUPPORTED
    assert f(byref(tables(max_rows=2000)), byref(j), A.POOL_SUM, FAKE, A.BF16, 3, 1, None) == INVALID_ARG
    assert f(byref(t), byref(j), A.POOL_SUM, None, A.BF16, 3, 1, None) == INVALID_ARG  # null X
    # valid no-ops: B = 0, F = 0
    assert f(byref(t), byref(bags(B=0, nnz=0)), A.POOL_SUM, None, A.BF16, 3, 1, None) == OK
    assert f(byref(t), byref(bags(F=0, nnz=0)), A.POOL_SUM, None, A.BF16, 3, 1, None) == OK


def _grad_out():
    return A.lattice_sparse_grad(unique_rows=FAKE, seg_offsets=FAKE, sorted_bags=FAKE,
                                 num_unique=FAKE, grad_rows=None)


def test_embbag_bwd_statuses(lib):
    t, j, out = tables(), bags(nnz=10), _grad_out()
    need = lib.lattice_embbag_bwd_workspace(byref(t), byref(j))
    assert need > 0
    f = lib.lattice_embbag_bwd
    args = lambda **k: (byref(k.get("t", t)), byref(k.get("j", j)), A.POOL_SUM, k.get("dX", FAKE),
                        A.BF16, k.get("n", 3), 1, k.get("out", byref(out)), 0.0, FAKE,
                        k.get("ws", need), None)
    assert f(*args(ws=need - 1)) == WORKSPACE
    assert "workspace" in last_error(lib)
    assert f(*args(out=None)) == INVALID_ARG
    bad = _grad_out()
    bad.seg_offsets = None
    assert f(*args(out=byref(bad))) == INVALID_ARG
    assert f(*args(dX=None)) == INVALID_ARG
    assert f(*args(n=2)) == INVALID_ARG
    assert f(*args(t=tables(dim=20))) == UNSUPPORTED
    # dX of B * n_slots * dim elements larger than 4 GiB
    big = bags(B=1 << 20, nnz=10)
    assert f(*args(j=big, n=1025, ws=lib.lattice_embbag_bwd_workspace(byref(t), byref(big)))) == UNSUPPORTED
    assert "4 GiB" in last_error(lib)


def test_validate_batch_statuses(lib):
    t, j = tables(), bags()
    first_bad = ctypes.c_int64(0)
    assert lib.lattice_validate_batch(byref(t), byref(j), None, None) == INVALID_ARG
    assert lib.lattice_validate_batch(None, byref(j), byref(first_bad), None) == INVALID_ARG
    assert lib.lattice_validate_batch(byref(t), byref(bags(B=0, nnz=0)), byref(first_bad), None) == OK
    assert first_bad.value == 0


# ---------------------------------------------------------------- interaction
def interact_desc(kind=A.FM, dtype=A.BF16, n=65, dim=128, rank=32, W=FAKE, layers=None, n_layers=0,
                  stack_n=0, eps=1e-5, emit=1):
    return A.lattice_interact_desc(kind=kind, dtype=dtype, n=n, dim=dim, rank=rank, emit_slot0=emit,
                                   fm_W=W, fm_dW=FAKE, n_layers=n_layers, stack_n=stack_n,
                                   ln_eps=eps, layers=layers)


def test_interact_statuses(lib):
    f = lib.lattice_interact_fwd
    d = interact_desc()
    assert f(None, 8, FAKE, FAKE, 1 << 20, None, 0, None) == INVALID_ARG
    assert f(byref(interact_desc(W=None)), 8, FAKE, FAKE, 1 << 20, None, 0, None) == INVALID_ARG
    assert f(byref(interact_desc(dim=12)), 8, FAKE, FAKE, 1 << 20, None, 0, None) == UNSUPPORTED
    assert f(byref(interact_desc(kind=7)), 8, FAKE, FAKE, 1 << 20, None, 0, None) == UNSUPPORTED
    # output row stride shorter than the row
    assert f(byref(d), 8, FAKE, FAKE, 100, None, 0, None) == INVALID_ARG
    assert "out_stride" in last_error(lib)
    assert f(byref(d), 8, None, FAKE, 1 << 20, None, 0, None) == INVALID_ARG
    assert f(byref(d), 0, None, None, 0, None, 0, None) == OK                    # B = 0: nothing to write
    # the stacked interaction: fp32 unsupported, missing layers, small workspace
    lay = (A.lattice_stack_layer * 1)(A.lattice_stack_layer(W=FAKE, A=FAKE, C=None, gamma=FAKE,
                                                            dW=FAKE, dA=FAKE, dC=None, dgamma=FAKE))
    st = interact_desc(kind=A.STACK, n=64, rank=64, layers=lay, n_layers=1, stack_n=64, emit=0, W=None)
    need = lib.lattice_interact_workspace(byref(st), 16)
    assert need > 0
    assert f(byref(st), 16, FAKE, FAKE, 64 * 128, FAKE, need - 1, None) == WORKSPACE
    st32 = interact_desc(kind=A.STACK, dtype=A.F32, n=64, rank=64, layers=lay, n_layers=1, stack_n=64,
                         emit=0, W=None)
    assert f(byref(st32), 16, FAKE, FAKE, 64 * 128, FAKE, need, None) == UNSUPPORTED
    st0 = interact_desc(kind=A.STACK, n=64, rank=64, layers=None, n_layers=0, stack_n=64, emit=0, W=None)
    assert f(byref(st0), 16, FAKE, FAKE, 64 * 128, FAKE, need, None) == INVALID_ARG
    # STACK layer 0 must have C when the vector count changes
    stc = interact_desc(kind=A.STACK, n=128, rank=64, layers=lay, n_layers=1, stack_n=64, emit=0, W=None)
    assert f(byref(stc), 16, FAKE, FAKE, 64 * 128, FAKE, 1 << 30, None) == INVALID_ARG
    # the DOT slot mask: DOT only, n <= 128, 16-byte aligned
    fm_mask = interact_desc()
    fm_mask.slot_mask = FAKE
    assert f(byref(fm_mask), 8, FAKE, FAKE, 1 << 20, None, 0, None) == INVALID_ARG
    assert "slot_mask" in last_error(lib)
    big = interact_desc(kind=A.DOT, n=129, dim=64, W=None)
    big.slot_mask = FAKE
    assert f(byref(big), 8, FAKE, FAKE, 1 << 20, None, 0, None) == INVALID_ARG
    odd = interact_desc(kind=A.DOT, n=97, dim=128, W=None)
    odd.slot_mask = FAKE + 4
    assert f(byref(odd), 8, FAKE, FAKE, 1 << 20, None, 0, None) == INVALID_ARG
    fm_fp8 = interact_desc()
    fm_fp8.fp8_proj = 2
    assert f(byref(fm_fp8), 8, FAKE, FAKE, 1 << 20, None, 0, None) == INVALID_ARG
    assert "fp8_proj" in last_error(lib)
    # the stacked interaction's saved state: offsets per layer, the last output the caller's
    stt = A.lattice_stack_state()
    assert lib.lattice_interact_state(byref(st), 16, byref(stt)) == OK
    assert stt.P[0] >= 0 and stt.F[0] > stt.P[0] and stt.H[0] > stt.F[0] and stt.Xn[0] == -1 and stt.P[1] == -1
    assert lib.lattice_interact_state(byref(interact_desc()), 16, byref(stt)) == OK and stt.P[0] == -1
    assert lib.lattice_interact_state(byref(st), 16, None) == INVALID_ARG
    fm_skip = interact_desc()
    fm_skip.skip_absent = 1
    assert f(byref(fm_skip), 8, FAKE, FAKE, 1 << 20, None, 0, None) == INVALID_ARG
    assert "skip_absent" in last_error(lib)
    # backward without the FM weight gradient
    nog = interact_desc()
    nog.fm_dW = None
    assert lib.lattice_interact_bwd(byref(nog), 8, FAKE, FAKE, 1 << 20, FAKE, FAKE, 1 << 30, None) == INVALID_ARG


# ---------------------------------------------------------------------- MLPs
def mlp(dims, dtype=A.BF16, relu_last=0):
    arr = (A.lattice_linear * (len(dims) - 1))(*[
        A.lattice_linear(in_dim=dims[i], out_dim=dims[i + 1], W=FAKE, b=FAKE, dW=FAKE, db=FAKE)
        for i in range(len(dims) - 1)])
    d = A.lattice_mlp_desc(dtype=dtype, n_layers=len(dims) - 1, layers=arr, relu_last=relu_last)
    d._keep = arr
    return d


def test_mlp_statuses(lib):
    d = mlp([64, 32, 4])
    acts = (ctypes.c_void_p * 2)(FAKE, FAKE)
    strides = (ctypes.c_int64 * 2)(32, 4)
    loss = A.lattice_loss_desc(labels=FAKE, mask=FAKE, loss=FAKE, d_logits=FAKE, d_logits_op=None)
    need = lib.lattice_mlp_heads_workspace(byref(d), 16)
    f = lib.lattice_mlp_heads_fwd
    assert f(byref(d), 16, FAKE, 64, acts, strides, byref(loss), FAKE, 0, None) == WORKSPACE
    assert f(byref(d), 16, FAKE, 63, acts, strides, None, FAKE, need, None) == INVALID_ARG  # in_stride
    bad = mlp([64, 32, 4])
    bad.layers[1].in_dim = 31
    assert f(byref(bad), 16, FAKE, 64, acts, strides, None, FAKE, need, None) == INVALID_ARG
    assert "in_dim" in last_error(lib)
    too_deep = mlp([8] * 10)
    assert f(byref(too_deep), 16, FAKE, 8, acts, strides, None, FAKE, need, None) == INVALID_ARG
    relu = mlp([64, 32, 4], relu_last=1)
    assert f(byref(relu), 16, FAKE, 64, acts, strides, byref(loss), FAKE, need, None) == INVALID_ARG
    b = lib.lattice_mlp_heads_bwd
    assert b(byref(d), 16, FAKE, 64, acts, strides, FAKE, 4, None, 0, FAKE, need - 1, None) == WORKSPACE
    assert b(byref(d), 16, FAKE, 64, acts, strides, FAKE, 3, None, 0, FAKE, need, None) == INVALID_ARG


# ------------------------------------------------------------- whole step
def model(dim=128, bottom_out=128, top_in=None, F=4, dense_in=16):
    n = F + 1
    top_in = top_in if top_in is not None else dim + n * 8
    m = A.lattice_model_desc(dtype=A.BF16, pool=A.POOL_SUM, tables=tables(dim=dim, max_rows=100),
                             num_features=F, dense_in=dense_in, bottom=mlp([dense_in, 64, bottom_out], relu_last=1),
                             interact=interact_desc(n=n, dim=dim, rank=8),
                             top=mlp([top_in, 64, 4]))
    m._keep = (m.bottom, m.top)
    return m


def step_opts(**k):
    return A.lattice_step_opts(lr_tables=0.0, emit_grad_rows=0, nnz_capacity=k.get("cap", 0))


def test_step_statuses(lib):
    m = model()
    lay = A.lattice_step_layout()
    o = step_opts()
    assert lib.lattice_step_plan(byref(m), 64, 1000, byref(o), byref(lay)) == OK
    assert lay.total_bytes > 0 and lay.X >= 0 and lay.dX > lay.X
    assert lay.top_grad[1] == lay.d_logits_op and lay.top_grad[0] >= 0 and lay.top_grad[2] == -1
    assert lay.bottom_grad[0] >= 0 and lay.bottom_grad[1] >= 0 and lay.bottom_grad[2] == -1
    batch = A.lattice_batch_desc(bags=bags(F=4, B=64, nnz=1000), dense=FAKE, labels=FAKE, mask=FAKE)
    s = lib.lattice_step
    assert s(byref(m), byref(batch), byref(o), FAKE, lay.total_bytes - 1, None) == WORKSPACE
    assert s(byref(m), byref(batch), byref(o), None, lay.total_bytes, None) == WORKSPACE
    # more lookups than the workspace was planned for
    assert s(byref(m), byref(batch), byref(step_opts(cap=999)), FAKE, 1 << 40, None) == INVALID_ARG
    assert "nnz_capacity" in last_error(lib)
    # model inconsistencies
    for bad in (model(bottom_out=64), model(top_in=100)):
        assert lib.lattice_step_plan(byref(bad), 64, 1000, byref(o), byref(lay)) == INVALID_ARG
    assert lib.lattice_step_plan(byref(model(dim=100, bottom_out=100)), 64, 1000, byref(o), byref(lay)) == UNSUPPORTED
    # feature count of the batch differs from the model's
    b2 = A.lattice_batch_desc(bags=bags(F=3, B=64, nnz=1000), dense=FAKE, labels=FAKE, mask=FAKE)
    assert s(byref(m), byref(b2), byref(o), FAKE, 1 << 40, None) == INVALID_ARG
    # null labels (the forward alone reads none; an empty batch: nothing to do)
    b3 = A.lattice_batch_desc(bags=bags(F=4, B=64, nnz=1000), dense=FAKE, labels=None, mask=FAKE)
    assert s(byref(m), byref(b3), byref(o), FAKE, 1 << 40, None) == INVALID_ARG
    fw = lib.lattice_forward
    assert fw(None, byref(b3), byref(o), FAKE, 1 << 40, None) == INVALID_ARG
    assert fw(byref(m), byref(b3), byref(o), FAKE, lay.total_bytes - 1, None) == WORKSPACE
    b0 = A.lattice_batch_desc(bags=bags(F=4, B=0, nnz=0), dense=None, labels=None, mask=None)
    assert fw(byref(m), byref(b0), byref(o), FAKE, 1 << 40, None) == OK
    # a side stream without its events
    o2 = step_opts()
    o2.side_stream = FAKE
    assert s(byref(m), byref(batch), byref(o2), FAKE, 1 << 40, None) == INVALID_ARG
    assert "side_events" in last_error(lib)
    evs = (ctypes.c_void_p * A.SIDE_EVENTS)(*([FAKE] * (A.SIDE_EVENTS - 1) + [None]))
    o2.side_events = ctypes.cast(evs, ctypes.POINTER(ctypes.c_void_p))
    assert s(byref(m), byref(batch), byref(o2), FAKE, 1 << 40, None) == INVALID_ARG
    # an empty batch plans a valid workspace (the step itself, which zeroes
    # the gradients, is a GPU test)
    assert lib.lattice_step_plan(byref(m), 0, 0, byref(o), byref(lay)) == OK
    assert lib.lattice_step(None, byref(batch), byref(o), FAKE, 1, None) == INVALID_ARG
