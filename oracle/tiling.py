"""Thread-block arrangements and the SDDMM cost model of section 7, in plain
Python over sets of points (oracle; test infrastructure only; small masks).

Section 7.2 defines a thread-block of m x n threads by an anchor t and a
stretch s; it computes the points t + (i*s, j*s) for i < m, j < n, and covers
those of them that lie in the mask's point set P.  For an arrangement of
lambda blocks that covers P it defines

* divergent threads  phi_TD = |(union of the computed points) - P|,
* redundant threads  phi_R  = lambda*m*n - |P| - phi_TD,
* reuse              phi_RU = |P| / (lambda*m*n),
* coalescing         phi_CMR = mean over the blocks of 1/stretch,
* cost               lambda / phi_CMR.

Section 7.3 (Algorithm 1, poset tiling) builds an arrangement in rounds: the
points of the uncovered set that no other uncovered point comes before
((x', y') comes before (x, y) when x' <= x and y' <= y) become anchors, and
the points their blocks compute leave the uncovered set, until it is empty.
Reading: the printed update of the uncovered set is garbled; here each round
removes every point the round's new blocks compute from the uncovered set.

Section 7.3.1 selects the stretch: 1 for polygonal masks; for a strided mask
of stride X the stretch minimising lambda * s over the divisors of X.
Reading: a mask is strided when every row with two or more points is a single
affine run and all of them share one stride X > 1 (rows with one point fit
any stride).  Equal costs go to the arrangement with fewer blocks (higher
reuse): in the section's worked example the stretched and the unstretched
arrangements of a stride-2 mask cost the same, and the text presents the
stretched one as the better.

Naive Tiling (Appendix C, the comparison point of the SDDMM tiling ablation
in section 10) cuts the mask into patches of m consecutive rows, starting at
row 0, and tiles each patch from left to right with unstretched m x n blocks:
the first block starts at the patch's leftmost point, the blocks follow each
other n columns apart, and a patch of width w (leftmost to rightmost point,
inclusive) takes ceil(w / n) of them.  Appendix C counts
lambda_naive = sum over patches of ceil(w / n) and gives its closed form for
structured dense polygons.

The grid arrangement (a second, separately labelled comparison) places
unstretched blocks at every multiple of (m, n) whose block meets P.
"""
from __future__ import annotations

from typing import Dict, Iterable, List, Set, Tuple

import numpy as np

from . import acsr as oacsr

Point = Tuple[int, int]


def points_of(mask: np.ndarray) -> Set[Point]:
    rows, cols = np.nonzero(np.asarray(mask, dtype=bool))
    return set(zip(rows.tolist(), cols.tolist()))


def comes_before(p: Point, q: Point) -> bool:
    """p comes before q: both coordinates of p are at most those of q."""
    return p[0] <= q[0] and p[1] <= q[1]


def minimal_set(uncovered: Set[Point]) -> List[Point]:
    """The points of `uncovered` that no other uncovered point comes before,
    by the definition (every pair compared), in (row, column) order."""
    pts = sorted(uncovered)
    out = []
    for p in pts:
        if not any(q != p and comes_before(q, p) for q in pts):
            out.append(p)
    return out


def computed(anchor: Point, m: int, n: int, s: int) -> Set[Point]:
    x, y = anchor
    return {(x + i * s, y + j * s) for i in range(m) for j in range(n)}


def poset_tiling(P: Set[Point], m: int, n: int, s: int):
    """Anchors in placement order (round by round, rows ascending) and the
    number of rounds."""
    uncovered = set(P)
    anchors: List[Point] = []
    rounds = 0
    while uncovered:
        top = minimal_set(uncovered)
        anchors.extend(top)
        for a in top:
            uncovered -= computed(a, m, n, s)
        rounds += 1
    return anchors, rounds


def naive_tiling(P: Set[Point], L: int, m: int, n: int) -> List[Point]:
    """Appendix C's Naive Tiling: anchors patch by patch (rows x0 = 0, m, 2m,
    ...), left to right inside each patch."""
    out = []
    for x0 in range(0, L, m):
        cols = [c for (r, c) in P if x0 <= r < x0 + m]
        if not cols:
            continue
        left, right = min(cols), max(cols)
        width = right - left + 1
        for k in range(-(-width // n)):
            out.append((x0, left + k * n))
    return out


def structured_polygon(r: int, h: int, l: int, lp: int) -> Set[Point]:
    """Appendix C's structured dense polygon with parameters (r, l, h, l'):
    r slabs of h rows; row y holds the l columns starting at floor(y/h)*l'.
    Points as (row, column)."""
    return {(y, (y // h) * lp + t) for y in range(r * h) for t in range(l)}


def grid_tiling(P: Set[Point], L: int, m: int, n: int) -> List[Point]:
    out = []
    for x in range(0, L, m):
        for y in range(0, L, n):
            if any((x + i, y + j) in P for i in range(m) for j in range(n)):
                out.append((x, y))
    return out


def metrics(P: Set[Point], anchors: Iterable[Point], m: int, n: int, s: int) -> Dict[str, float]:
    anchors = list(anchors)
    lam = len(anchors)
    comp: Set[Point] = set()
    for a in anchors:
        comp |= computed(a, m, n, s)
    assert P <= comp, "the arrangement covers the point set"
    td = len(comp - P)
    return {"blocks": lam, "points": len(P), "divergent": td,
            "redundant": lam * m * n - len(P) - td,
            "reuse": len(P) / (lam * m * n) if lam else 1.0,
            "coalesced": 1.0 / s, "cost": lam * s, "stretch": s}


def common_stride(mask: np.ndarray) -> int:
    """X when every row of two or more points is one affine run of the
    common stride X > 1, else 1."""
    X = None
    for row in np.asarray(mask, dtype=bool):
        cols = np.nonzero(row)[0].tolist()
        if len(cols) < 2:
            continue
        ab = oacsr.affine_indices(cols)
        if ab is None:
            return 1
        stride = int(1 / ab[0])
        if stride == 1:
            return 1
        if X is None:
            X = stride
        elif stride != X:
            return 1
    return X if X else 1


def poset_with_selection(mask: np.ndarray, m: int, n: int):
    """Poset tiling with the selected stretch: (anchors, rounds, metrics)."""
    P = points_of(mask)
    X = common_stride(mask)
    best = None
    for s in range(1, X + 1):
        if X % s:
            continue
        anchors, rounds = poset_tiling(P, m, n, s)
        met = metrics(P, anchors, m, n, s)
        if best is None or met["cost"] < best[2]["cost"] or (
                met["cost"] == best[2]["cost"] and met["blocks"] < best[2]["blocks"]):
            best = (anchors, rounds, met)
    return best
