"""The paper's ACSR definitions, exactly (oracle; test infrastructure only).

All arithmetic is on ``fractions.Fraction`` so the real-valued affine indices
of the paper are represented without rounding.

* Definition 1 (section 4.1): a point set {(x_1, y), ..., (x_k, y)} sorted by
  x is affine-compressible iff some real a, b satisfy
  x_t * a + b + 1 = x_{t+1} * a + b for every consecutive pair, i.e. the
  affine map s = a * x + b sends the points to consecutive integers.
* Section 5.1: the affine indices of a row come from its first two columns
  i0 < i1 by solving [[i0, 1], [i1, 1]] [a, b]^T = [0, 1]^T; the row is then
  verified point by point with the same consecutive-pair equation.  A mask is
  regular iff every row is affine-compressible (section 4.1).
* Section 5.1: a value at compressed position sparse_i of a row with affine
  indices (a, b) sits at dense column (sparse_i - b) / a.
* Section 5.2 ("fast indexing"): membership of dense column j in a row is
  decided from (a, b, nnzs) in O(1).  The printed predicate is garbled (it
  ignores the upper end of the row and mixes index units); the reading used
  here is the one the construction implies: j belongs to the row iff a*j + b
  is an integer in [0, nnzs).

Readings where the paper is silent: a row with a single point has no second
point to solve with; it is given a = 1, b = -x_1 (so its one value sits at
sparse index 0).  An empty row is given a = 1, b = 0, nnzs = 0.
"""
from __future__ import annotations

from fractions import Fraction
from typing import Optional, Sequence, Tuple

import numpy as np


def solve_affine_indices(i0: int, i1: int) -> Tuple[Fraction, Fraction]:
    """Solve [[i0, 1], [i1, 1]] [a, b]^T = [0, 1]^T exactly (section 5.1)."""
    det = Fraction(i0) * 1 - Fraction(1) * i1          # i0 - i1
    if det == 0:
        raise ZeroDivisionError("two equal columns do not determine (a, b)")
    # Cramer's rule on the 2x2 system.
    a = (Fraction(0) * 1 - Fraction(1) * 1) / det       # (0*1 - 1*1) / (i0 - i1)
    b = (Fraction(i0) * 1 - Fraction(i1) * 0) / det     # (i0*1 - i1*0) / (i0 - i1)
    return a, b


def consecutive(x_prev: int, x_next: int, a: Fraction, b: Fraction) -> bool:
    """The per-pair condition of Definition 1: x_prev*a + b + 1 == x_next*a + b."""
    return Fraction(x_prev) * a + b + 1 == Fraction(x_next) * a + b


def affine_indices(cols: Sequence[int]) -> Optional[Tuple[Fraction, Fraction]]:
    """(a, b) of an ascending column list, or None if not affine-compressible."""
    cols = [int(c) for c in cols]
    if len(cols) == 0:
        return Fraction(1), Fraction(0)
    if len(cols) == 1:
        return Fraction(1), Fraction(-cols[0])
    a, b = solve_affine_indices(cols[0], cols[1])
    for t in range(1, len(cols)):
        if not consecutive(cols[t - 1], cols[t], a, b):
            return None
    return a, b


def is_affine_compressible(points: Sequence[Tuple[int, int]]) -> bool:
    """Definition 1 on a point set of one row (points are (x, y) pairs)."""
    xs = sorted(int(x) for x, _ in points)
    return affine_indices(xs) is not None


def is_regular(mask: np.ndarray) -> bool:
    """Every row's point set is affine-compressible (section 4.1)."""
    mask = np.asarray(mask, dtype=bool)
    return all(affine_indices(np.nonzero(row)[0]) is not None for row in mask)


def dense_col(sparse_i: int, a: Fraction, b: Fraction) -> Fraction:
    """Dense column of the value at compressed position sparse_i (section 5.1)."""
    return (Fraction(sparse_i) - b) / a


def sparse_index(dense_j: int, a: Fraction, b: Fraction) -> Fraction:
    """Compressed position a * j + b of dense column j (inverse of dense_col)."""
    return a * dense_j + b


def contains(dense_j: int, a: Fraction, b: Fraction, nnzs: int) -> bool:
    """O(1) membership of column j in a row (section 5.2, as read above)."""
    s = sparse_index(dense_j, a, b)
    return s.denominator == 1 and 0 <= s < nnzs
