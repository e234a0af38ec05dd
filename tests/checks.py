"""Checkers shared by the oracle pins and the device parity tests.

These encode properties that pin a result without a second implementation:
the characterization of max/argmax, the invariants of a stable
destination-major CSR, and the summand-scaled error used for sums.
"""
from __future__ import annotations

import numpy as np


def check_max_characterization(rowptr, col, x_f32, w, out_max, argmax, rows=None,
                               chunk_edges=1 << 22):
    """Unique characterization of (max, argmax) per (row, feature): argmax is
    the first CSR position p in the row whose message equals the row maximum
    (values compared as numbers, so -0.0 == +0.0), and out_max holds that
    message's bits.  Empty rows give (+0.0, -1).  `rows` lists which row each
    output row is (default: all rows in order).  Raises AssertionError."""
    rowptr = np.asarray(rowptr, np.int64)
    rows = np.arange(rowptr.shape[0] - 1) if rows is None else np.asarray(rows, np.int64)
    out_max = np.asarray(out_max, np.float32)
    argmax = np.asarray(argmax, np.int64)
    assert out_max.shape == argmax.shape and out_max.shape[0] == rows.shape[0]
    deg = rowptr[rows + 1] - rowptr[rows]
    empty = deg == 0
    assert np.all(argmax[empty] == -1), "empty row with argmax != -1"
    assert np.all(out_max[empty].view(np.uint32) == 0), "empty row with max != +0.0"
    ks = np.nonzero(~empty)[0]
    i = 0
    while i < ks.shape[0]:
        # take rows until about chunk_edges edges are gathered
        j = i
        tot = 0
        while j < ks.shape[0] and (j == i or tot + deg[ks[j]] <= chunk_edges):
            tot += deg[ks[j]]
            j += 1
        kk = ks[i:j]
        starts_g = rowptr[rows[kk]]
        d = deg[kk]
        # global CSR positions of every edge of these rows, row after row
        offs = np.concatenate([[0], np.cumsum(d)[:-1]])
        pos = np.repeat(starts_g - offs, d) + np.arange(int(d.sum()))
        m = _row_messages(np.asarray(col)[pos], x_f32, None if w is None else np.asarray(w)[pos])
        mx = np.maximum.reduceat(m, offs, axis=0)
        rep = np.repeat(np.arange(kk.shape[0]), d)
        big = np.iinfo(np.int64).max
        cand = np.where(m == mx[rep], pos[:, None], big)
        first = np.minimum.reduceat(cand, offs, axis=0)
        bad = first != argmax[kk]
        if np.any(bad):
            a, f = np.argwhere(bad)[0]
            raise AssertionError(f"row {rows[kk[a]]} feature {f}: argmax {argmax[kk[a], f]}, "
                                 f"expected {first[a, f]}")
        at = m[first - np.repeat(starts_g - offs, 1)[:, None], np.arange(m.shape[1])[None, :]]
        if not np.array_equal(at.view(np.uint32), out_max[kk].view(np.uint32)):
            a, f = np.argwhere(at.view(np.uint32) != out_max[kk].view(np.uint32))[0]
            raise AssertionError(f"row {rows[kk[a]]} feature {f}: max bits differ from the "
                                 f"message at argmax")
        i = j


def _row_messages(col_row, x_f32, w_row):
    """fp32 messages of one row's edges: x[col] or fl32(w * x[col])."""
    m = x_f32[col_row.astype(np.int64)]
    if w_row is not None:
        m = (w_row.astype(np.float64)[:, None] * m.astype(np.float64)).astype(np.float32)
    return m


def check_csr_invariants(src, dst, n_dst, rowptr, col, perm):
    """rowptr[0]=0, rowptr[N]=E, monotone, diff = in-degree; perm is a
    permutation, strictly increasing within each row, and maps each CSR slot
    back to its COO edge (col = src[perm], row = dst[perm])."""
    src, dst = np.asarray(src), np.asarray(dst)
    rowptr = np.asarray(rowptr, np.int64)
    perm = np.asarray(perm, np.int64)
    E = src.shape[0]
    assert rowptr.shape == (n_dst + 1,)
    assert rowptr[0] == 0 and rowptr[-1] == E
    assert np.all(np.diff(rowptr) >= 0)
    assert np.array_equal(np.diff(rowptr), np.bincount(dst, minlength=n_dst))
    assert np.array_equal(np.sort(perm), np.arange(E))
    assert np.array_equal(np.asarray(col), src[perm])
    row_of = np.repeat(np.arange(n_dst), np.diff(rowptr))
    assert np.array_equal(dst[perm], row_of)
    if E > 1:
        same = row_of[1:] == row_of[:-1]
        assert np.all(perm[1:][same] > perm[:-1][same]), "not stable within a row"


def scaled_error(y, ref, scale):
    """max |y - ref| / scale; where scale == 0 the values must be equal."""
    y = np.asarray(y, np.float64)
    ref = np.asarray(ref, np.float64)
    scale = np.asarray(scale, np.float64)
    d = np.abs(y - ref)
    zero = scale == 0
    if np.any(d[zero] != 0):
        return float("inf")
    if not np.any(~zero):
        return 0.0
    return float(np.max(d[~zero] / scale[~zero]))
