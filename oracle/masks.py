"""Brute-force mask enumeration (oracle; test infrastructure only).

A mask M over an L x L attention matrix has M[i, j] = 1 when query row i
attends to key column j (section 4.1 maps M[i][j] to the point (j, i), so the
x coordinate is the column and y the row).  Each pattern is its defining
predicate, evaluated at every (i, j) -- O(L^2), no structure exploited.

The predicates restate the workload descriptions:

* window        |i - j| <= w
* blocked       j lies in the block of i or in the block before it (block 0
                has no predecessor)
* strided_local causal: j in [i - local + 1, i], or (j mod stride == stride - 1
                and j <= i); a column that satisfies both counts once
* dilated       j - i is a multiple of the dilation g and |j - i| <= g * w
* window_global |i - j| <= w, or i < G (global rows), or j < G (global columns)
* full          every (i, j)
"""
from __future__ import annotations

from typing import Callable, Dict, List

import numpy as np


def predicate(kind: str, params: Dict[str, int]) -> Callable[[int, int], bool]:
    """Scalar predicate M(i, j) -> bool for a pattern."""
    p = dict(params)
    if kind == "window":
        w = p["w"]
        return lambda i, j: abs(i - j) <= w
    if kind == "blocked":
        b = p["block"]
        return lambda i, j: (j // b) == (i // b) or (j // b) == (i // b) - 1
    if kind == "strided_local":
        n, s = p["local"], p["stride"]
        return lambda i, j: (i - n < j <= i) or (j % s == s - 1 and j <= i)
    if kind == "dilated":
        w, g = p["w"], p["dilation"]
        return lambda i, j: (j - i) % g == 0 and abs(j - i) <= g * w
    if kind == "window_global":
        w, G = p["w"], p["n_global"]
        return lambda i, j: abs(i - j) <= w or i < G or j < G
    if kind == "full":
        return lambda i, j: True
    raise ValueError(f"unknown pattern kind {kind!r}")


def dense_mask(kind: str, params: Dict[str, int], L: int) -> np.ndarray:
    """Boolean [L, L] mask, the predicate evaluated on the full (i, j) grid."""
    p = dict(params)
    i = np.arange(L, dtype=np.int64)[:, None]
    j = np.arange(L, dtype=np.int64)[None, :]
    if kind == "window":
        m = np.abs(i - j) <= p["w"]
    elif kind == "blocked":
        b = p["block"]
        m = ((j // b) == (i // b)) | ((j // b) == (i // b) - 1)
    elif kind == "strided_local":
        n, s = p["local"], p["stride"]
        m = ((j > i - n) & (j <= i)) | ((j % s == s - 1) & (j <= i))
    elif kind == "dilated":
        w, g = p["w"], p["dilation"]
        m = ((j - i) % g == 0) & (np.abs(j - i) <= g * w)
    elif kind == "window_global":
        w, G = p["w"], p["n_global"]
        m = (np.abs(i - j) <= w) | (i < G) | (j < G)
    elif kind == "full":
        m = np.ones((L, L), dtype=bool)
    else:
        raise ValueError(f"unknown pattern kind {kind!r}")
    return np.array(np.broadcast_to(m, (L, L)), dtype=bool, copy=True)


def dense_mask_loops(kind: str, params: Dict[str, int], L: int) -> np.ndarray:
    """Same mask from the scalar predicate with plain Python loops (small L)."""
    f = predicate(kind, params)
    m = np.zeros((L, L), dtype=bool)
    for i in range(L):
        for j in range(L):
            m[i, j] = f(i, j)
    return m


def csr(mask: np.ndarray):
    """(row_ptr int64[L+1], col_idx int64[nnz]) of a boolean mask.

    Columns are listed in ascending order within each row: the order the
    row-compressed row-major ACSR layout stores a row's values in (section 5.1).
    """
    mask = np.asarray(mask, dtype=bool)
    counts = mask.sum(axis=1).astype(np.int64)
    row_ptr = np.zeros(mask.shape[0] + 1, dtype=np.int64)
    np.cumsum(counts, out=row_ptr[1:])
    col_idx = np.nonzero(mask)[1].astype(np.int64)   # row-major traversal
    return row_ptr, col_idx


def csc(mask: np.ndarray):
    """(col_ptr int64[L+1], row_idx int64[nnz]) of a boolean mask: rows in
    ascending order within each column, column by column -- the order the
    column-compressed column-major layout stores the values in (section 5.2).
    Traverses the mask column by column (Fortran order)."""
    mask = np.asarray(mask, dtype=bool)
    counts = mask.sum(axis=0).astype(np.int64)
    col_ptr = np.zeros(mask.shape[1] + 1, dtype=np.int64)
    np.cumsum(counts, out=col_ptr[1:])
    cols_major = np.nonzero(mask.T)                      # (column, row) pairs, column-major
    row_idx = cols_major[1].astype(np.int64)
    return col_ptr, row_idx


def colmajor_source(mask: np.ndarray) -> np.ndarray:
    """For every slot of the column-major value order, the CSR (row-major)
    position of the same (row, column) entry: colmajor = csr_values[this]."""
    mask = np.asarray(mask, dtype=bool)
    pos = np.full(mask.shape, -1, dtype=np.int64)
    pos[mask] = np.arange(int(mask.sum()), dtype=np.int64)  # row-major numbering
    return pos.T[mask.T]                                     # read back column by column


def row_columns(kind: str, params: Dict[str, int], L: int, i: int) -> np.ndarray:
    """Ascending key columns of one row, by brute force over every j."""
    f = predicate(kind, params)
    return np.array([j for j in range(L) if f(i, j)], dtype=np.int64)


def row_columns_fast(kind: str, params: Dict[str, int], L: int, rows) -> List[np.ndarray]:
    """Ascending columns of several rows, the predicate vectorised over j."""
    out = []
    j = np.arange(L, dtype=np.int64)
    for i in rows:
        m = dense_mask_row(kind, params, L, int(i), j)
        out.append(np.nonzero(m)[0].astype(np.int64))
    return out


def dense_mask_row(kind, params, L, i, j=None) -> np.ndarray:
    p = dict(params)
    if j is None:
        j = np.arange(L, dtype=np.int64)
    if kind == "window":
        return np.abs(i - j) <= p["w"]
    if kind == "blocked":
        b = p["block"]
        return ((j // b) == (i // b)) | ((j // b) == (i // b) - 1)
    if kind == "strided_local":
        n, s = p["local"], p["stride"]
        return ((j > i - n) & (j <= i)) | ((j % s == s - 1) & (j <= i))
    if kind == "dilated":
        w, g = p["w"], p["dilation"]
        return ((j - i) % g == 0) & (np.abs(j - i) <= g * w)
    if kind == "window_global":
        w, G = p["w"], p["n_global"]
        return (np.abs(i - j) <= w) | (i < G) | (j < G)
    if kind == "full":
        return np.ones(L, dtype=bool)
    raise ValueError(f"unknown pattern kind {kind!r}")


# --------------------------------------------------------------------------
# Masks given as a union of affine terms (the pattern-descriptor language of
# the library's C interface, which generalises the per-row affine index map
# of section 5.1 to row ranges and row groups).  Term t covers rows
# row_lo <= i < row_hi; with q = floor(i / group) * group its columns are
# j = j_lo(i) + stride * k for k >= 0 while j <= j_hi(i), where
# j_lo(i) = lo_i * i + lo_q * q + lo_c and j_hi(i) = hi_i * i + hi_q * q +
# hi_c, keeping only 0 <= j < L (clamping keeps the residue mod stride).
def terms_mask_loops(L: int, terms) -> np.ndarray:
    """The definition above, one term, row and column at a time."""
    M = np.zeros((L, L), dtype=bool)
    for t in terms:
        for i in range(t["row_lo"], t["row_hi"]):
            q = (i // t["group"]) * t["group"]
            lo = t["lo_i"] * i + t["lo_q"] * q + t["lo_c"]
            hi = t["hi_i"] * i + t["hi_q"] * q + t["hi_c"]
            for j in range(lo, hi + 1, t["stride"]):
                if 0 <= j < L:
                    M[i, j] = True
    return M


def terms_mask(L: int, terms) -> np.ndarray:
    """Same mask, each term evaluated on the whole (i, j) grid at once."""
    i = np.arange(L, dtype=np.int64)[:, None]
    j = np.arange(L, dtype=np.int64)[None, :]
    M = np.zeros((L, L), dtype=bool)
    for t in terms:
        q = (i // t["group"]) * t["group"]
        lo = t["lo_i"] * i + t["lo_q"] * q + t["lo_c"]
        hi = t["hi_i"] * i + t["hi_q"] * q + t["hi_c"]
        rows = (i >= t["row_lo"]) & (i < t["row_hi"])
        M |= rows & (j >= lo) & (j <= hi) & ((j - lo) % t["stride"] == 0)
    return M
