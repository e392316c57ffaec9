"""Pooled embedding lookup over jagged multi-hot features, its gradient, the
row bookkeeping of the sparse gradient and the row-sparse SGD update.

Test infrastructure only (see the package docstring).

Definitions (Section 3.3.1: categorical features go through embedding tables
and yield one d-vector per feature and sample, output shape (B, |F_c|, d);
Section 3.2: a feature a record does not carry is zero-padded, i.e. an empty
bag pools to the zero vector):

* Layout: bag ``f*B + b`` holds positions ``offsets[f*B+b] .. offsets[f*B+b+1]-1``
  of ``indices``; all tables live in one ``[total_rows, d]`` array and table
  ``f`` starts at global row ``row_base[f]``.
* Pool (sum):   ``pooled[b, f] = sum_{j in bag(f,b)} table[row_base[f] + indices[j]]``;
  pool (mean):  the same divided by the bag length (empty bag -> 0).
* Gradient:     ``G[r] = sum over occurrences j with global row r of
  dpooled[b(j), f(j)]`` (divided by the bag length for mean pooling); only rows
  that occur exist in the output.
* Bookkeeping:  key ``= row_base[f] + index``; unique keys ascending, their
  occurrence counts, exclusive-scan segment offsets, and the occurrences in
  key order with ties kept in position order.
* SGD:          ``E'[r] = round(E[r] - lr * G[r])`` for every occurring row,
  evaluated in float64 with one rounding to the storage dtype; other rows are
  untouched.
"""
import numpy as np


def bag_of_positions(offsets, F, B):
    """(bag id, feature, sample) of every position of ``indices``."""
    lengths = np.diff(np.asarray(offsets, dtype=np.int64))
    bag = np.repeat(np.arange(F * B, dtype=np.int64), lengths)
    return bag, bag // B, bag % B


def pool_forward(table, row_base, offsets, indices, F, B, mode="sum"):
    """Pooled vectors ``[B, F, d]`` in float64 (Section 3.3.1)."""
    table = np.asarray(table, dtype=np.float64)
    d = table.shape[1]
    bag, f, _ = bag_of_positions(offsets, F, B)
    rows = table[np.asarray(row_base, dtype=np.int64)[f] + np.asarray(indices, dtype=np.int64)]
    out = np.zeros((F * B, d), dtype=np.float64)
    np.add.at(out, bag, rows)
    if mode == "mean":
        lengths = np.diff(np.asarray(offsets, dtype=np.int64)).astype(np.float64)
        out /= np.maximum(lengths, 1.0)[:, None]
    elif mode != "sum":
        raise ValueError(mode)
    return out.reshape(F, B, d).transpose(1, 0, 2)


def row_keys(row_base, offsets, indices, F, B):
    """Global row id (int64) of every position."""
    _, f, _ = bag_of_positions(offsets, F, B)
    return np.asarray(row_base, dtype=np.int64)[f] + np.asarray(indices, dtype=np.int64)


def bookkeeping(row_base, offsets, indices, F, B):
    """Unique rows ascending, counts, segment offsets, sorted positions and
    their bag ids (ties in position order)."""
    keys = row_keys(row_base, offsets, indices, F, B)
    order = np.argsort(keys, kind="stable")
    uniq, first, counts = np.unique(keys[order], return_index=True, return_counts=True)
    bag, _, _ = bag_of_positions(offsets, F, B)
    return dict(unique_rows=uniq, counts=counts, seg_offsets=first,
                sorted_positions=order, sorted_bags=bag[order], keys=keys)


def pool_backward(dpooled, row_base, offsets, indices, F, B, mode="sum"):
    """Row-coalesced gradient: (unique rows ascending, G [U, d] float64)."""
    dpooled = np.asarray(dpooled, dtype=np.float64)        # [B, F, d]
    bag, f, b = bag_of_positions(offsets, F, B)
    contrib = dpooled[b, f]                                # [nnz, d]
    if mode == "mean":
        lengths = np.diff(np.asarray(offsets, dtype=np.int64)).astype(np.float64)
        contrib = contrib / lengths[bag][:, None]
    keys = row_keys(row_base, offsets, indices, F, B)
    uniq = np.unique(keys)
    G = np.zeros((uniq.size, dpooled.shape[2]), dtype=np.float64)
    np.add.at(G, np.searchsorted(uniq, keys), contrib)
    return uniq, G


def sgd_rows(E_rows, G, lr, rnd):
    """Updated values of the occurring rows: ``rnd(E - lr*G)``."""
    return rnd(np.asarray(E_rows, dtype=np.float64) - float(lr) * np.asarray(G, dtype=np.float64))
