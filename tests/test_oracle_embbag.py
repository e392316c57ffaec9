"""Pins for the oracle's pooled lookup, sparse gradient, bookkeeping and SGD."""
import collections

import numpy as np
import pytest

from oracle import embbag
from oracle.bf16 import round_bf16, identity


def _jagged(r, F, B, rows, max_len, allow_empty=True):
    lo = 0 if allow_empty else 1
    lens = r.integers(lo, max_len + 1, size=F * B)
    offsets = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    indices = r.integers(0, rows, size=int(offsets[-1])).astype(np.int32)
    row_base = np.arange(F + 1, dtype=np.int64) * rows
    return offsets, indices, row_base


def _count_matrix(offsets, indices, row_base, F, B, total_rows):
    """Dense one-hot count matrix C[bag, global_row] by explicit loops."""
    C = np.zeros((F * B, total_rows))
    for f in range(F):
        for b in range(B):
            bag = f * B + b
            for j in range(offsets[bag], offsets[bag + 1]):
                C[bag, row_base[f] + indices[j]] += 1
    return C


def test_single_index_bag_equals_row():
    r = np.random.default_rng(0)
    table = r.standard_normal((3 * 10, 4)).astype(np.float32)
    offsets = np.array([0, 1, 2, 3], np.int32)            # F=3, B=1, one index each
    indices = np.array([7, 0, 9], np.int32)
    row_base = np.array([0, 10, 20, 30])
    out = embbag.pool_forward(table, row_base, offsets, indices, 3, 1)
    for f in range(3):
        np.testing.assert_array_equal(out[0, f], table[row_base[f] + indices[f]].astype(np.float64))


def test_k_copies_and_empty_bag():
    table = np.arange(20, dtype=np.float64).reshape(5, 4)
    offsets = np.array([0, 6, 6], np.int32)               # F=1, B=2: bag0 six copies, bag1 empty
    indices = np.full(6, 3, np.int32)
    out = embbag.pool_forward(table, [0, 5], offsets, indices, 1, 2)
    np.testing.assert_array_equal(out[0, 0], 6 * table[3])
    np.testing.assert_array_equal(out[1, 0], np.zeros(4))


@pytest.mark.parametrize("mode", ["sum", "mean"])
def test_brute_force_count_matrix(mode):
    r = np.random.default_rng(2)
    F, B, rows, d = 3, 5, 7, 4
    offsets, indices, row_base = _jagged(r, F, B, rows, 6)
    table = r.standard_normal((F * rows, d))
    C = _count_matrix(offsets, indices, row_base, F, B, F * rows)
    if mode == "mean":
        C = C / np.maximum(C.sum(1, keepdims=True), 1)
    ref = (C @ table).reshape(F, B, d).transpose(1, 0, 2)
    out = embbag.pool_forward(table, row_base, offsets, indices, F, B, mode)
    np.testing.assert_allclose(out, ref, rtol=1e-13, atol=1e-13)


def test_linearity_in_table():
    r = np.random.default_rng(3)
    F, B, rows, d = 2, 4, 6, 3
    offsets, indices, row_base = _jagged(r, F, B, rows, 5)
    T1, T2 = r.standard_normal((F * rows, d)), r.standard_normal((F * rows, d))
    f = lambda T: embbag.pool_forward(T, row_base, offsets, indices, F, B)
    np.testing.assert_allclose(f(2 * T1 - 3 * T2), 2 * f(T1) - 3 * f(T2), atol=1e-12)


@pytest.mark.parametrize("mode", ["sum", "mean"])
def test_gradient_brute_force(mode):
    r = np.random.default_rng(4)
    F, B, rows, d = 3, 6, 5, 4
    offsets, indices, row_base = _jagged(r, F, B, rows, 5)
    dpooled = r.standard_normal((B, F, d))
    C = _count_matrix(offsets, indices, row_base, F, B, F * rows)
    if mode == "mean":
        C = C / np.maximum(C.sum(1, keepdims=True), 1)
    dflat = dpooled.transpose(1, 0, 2).reshape(F * B, d)
    full = C.T @ dflat                                    # gradient w.r.t. every table row
    uniq, G = embbag.pool_backward(dpooled, row_base, offsets, indices, F, B, mode)
    touched = np.flatnonzero(C.sum(0) > 0)
    np.testing.assert_array_equal(uniq, touched)
    np.testing.assert_allclose(G, full[touched], rtol=1e-12, atol=1e-12)
    # untouched rows have zero gradient in the dense form
    assert np.all(np.delete(full, touched, axis=0) == 0)


def test_gradient_sum_invariant():
    r = np.random.default_rng(5)
    F, B, rows, d = 4, 8, 9, 3
    offsets, indices, row_base = _jagged(r, F, B, rows, 7)
    dpooled = r.standard_normal((B, F, d))
    _, G = embbag.pool_backward(dpooled, row_base, offsets, indices, F, B)
    lens = np.diff(offsets).reshape(F, B)
    expect = np.einsum("fb,bfd->d", lens, dpooled)         # each bag contributes len * dpooled
    np.testing.assert_allclose(G.sum(0), expect, rtol=1e-12)


def test_bookkeeping_against_python_sort():
    r = np.random.default_rng(6)
    F, B, rows = 3, 7, 6
    offsets, indices, row_base = _jagged(r, F, B, rows, 6)
    bk = embbag.bookkeeping(row_base, offsets, indices, F, B)
    occ = []                                              # (key, position, bag) by loops
    for f in range(F):
        for b in range(B):
            for j in range(offsets[f * B + b], offsets[f * B + b + 1]):
                occ.append((int(row_base[f] + indices[j]), j, f * B + b))
    occ_sorted = sorted(occ)                              # key then position: a stable order
    cnt = collections.Counter(k for k, _, _ in occ)
    uniq = sorted(cnt)
    assert list(bk["unique_rows"]) == uniq
    assert list(bk["counts"]) == [cnt[k] for k in uniq]
    seg = [0]
    for k in uniq[:-1]:
        seg.append(seg[-1] + cnt[k])
    assert list(bk["seg_offsets"]) == seg
    assert list(bk["sorted_positions"]) == [j for _, j, _ in occ_sorted]
    assert list(bk["sorted_bags"]) == [bg for _, _, bg in occ_sorted]


def test_sgd_closed_form():
    E = np.array([[1.0, -2.0], [0.5, 0.25]])
    G = np.array([[10.0, 0.0], [-4.0, 2.0]])
    np.testing.assert_array_equal(embbag.sgd_rows(E, G, 0.5, identity), [[-4.0, -2.0], [2.5, -0.75]])
    # one rounding of the exact value: 1 - 2^-9 rounds (tie) to the even value 1.0
    out = embbag.sgd_rows(np.array([[1.0]]), np.array([[2.0 ** -9]]), 1.0, round_bf16)
    assert out[0, 0] == 1.0
