"""The tiling oracle (section 7) against the paper's worked example, the
definitions of section 7.2 and hand-derived minimal sets."""
import json
import os

import numpy as np
import pytest

from oracle import masks as om
from oracle import tiling as ot

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "poset_example.json")))


def _mask(points, L):
    M = np.zeros((L, L), dtype=bool)
    for x, y in points:
        M[x, y] = True
    return M


def test_worked_example_stretch_two():
    P = {tuple(p) for p in GOLD["points"]}
    anchors, _ = ot.poset_tiling(P, GOLD["m"], GOLD["n"], 2)
    g = GOLD["stretch2"]
    assert [list(a) for a in anchors] == g["anchors"]
    for a, cov in zip(anchors, g["covers"]):
        assert ot.computed(a, 2, 2, 2) & P == {tuple(c) for c in cov}
    met = ot.metrics(P, anchors, 2, 2, 2)
    assert met["reuse"] == g["reuse"] and met["coalesced"] == g["coalesced"]
    assert met["divergent"] == 0 and met["redundant"] == 0


def test_worked_example_stretch_one():
    P = {tuple(p) for p in GOLD["points"]}
    anchors, _ = ot.poset_tiling(P, 2, 2, 1)
    met = ot.metrics(P, anchors, 2, 2, 1)
    g = GOLD["stretch1"]
    for k in ("blocks", "divergent", "redundant", "reuse", "coalesced"):
        assert met[k] == g[k], k


def test_stretch_selection_on_worked_example():
    anchors, _, met = ot.poset_with_selection(_mask(GOLD["points"], 4), 2, 2)
    assert met["stretch"] == 2 and [list(a) for a in anchors] == GOLD["stretch2"]["anchors"]


def test_minimal_set_hand_derived():
    # (1,1) comes before (2,2) and (3,3); nothing comes before (0,3), (1,1), (2,0)
    P = {(0, 3), (1, 1), (2, 0), (2, 2), (3, 3)}
    assert ot.minimal_set(P) == [(0, 3), (1, 1), (2, 0)]
    # equal points in a column: the upper one comes before the lower
    assert ot.minimal_set({(0, 5), (4, 5)}) == [(0, 5)]
    assert ot.minimal_set({(2, 2)}) == [(2, 2)]


@pytest.mark.parametrize("kind,params,L,m,n", [
    ("window", {"w": 3}, 30, 4, 4), ("blocked", {"block": 5}, 23, 4, 8),
    ("dilated", {"w": 3, "dilation": 3}, 28, 3, 3), ("strided_local", {"local": 3, "stride": 5}, 25, 2, 4)])
def test_arrangement_definitions(kind, params, L, m, n):
    """Poset and grid arrangements cover the mask; anchors are distinct mask
    points (poset); the two forms of reuse in section 7.2 agree."""
    M = om.dense_mask(kind, params, L)
    P = ot.points_of(M)
    anchors, rounds, met = ot.poset_with_selection(M, m, n)
    assert len(set(anchors)) == len(anchors) and set(anchors) <= P and rounds >= 1
    lam, td, r = met["blocks"], met["divergent"], met["redundant"]
    assert r >= 0 and td >= 0
    assert abs(met["reuse"] - (m * n - td / lam - r / lam) / (m * n)) < 1e-12
    grid = ot.grid_tiling(P, L, m, n)
    gm = ot.metrics(P, grid, m, n, 1)
    assert gm["redundant"] == 0                       # grid blocks never overlap
    X = ot.common_stride(M)
    assert X == (params["dilation"] if kind == "dilated" else 1)
    costs = {s: ot.metrics(P, ot.poset_tiling(P, m, n, s)[0], m, n, s)["cost"]
             for s in range(1, X + 1) if X % s == 0}
    assert met["cost"] == min(costs.values()) and X % met["stretch"] == 0


# --------------------------------------------------------------------------
# Naive Tiling (Appendix C) pinned by its closed form for structured dense
# polygons, written out here case by case from the theorem's statement:
# with kappa = gcd(m, h), m = tau_m * kappa, h = tau_h * kappa and
# tau_m = alpha * tau_h + beta (0 <= beta < tau_h),
#   beta == 0: (r / tau_m) * tau_h * ceil((l + (alpha - 1) l') / n)
#   beta != 0: (r / tau_m) * ((beta - 1) ceil((l + (alpha + 1) l') / n)
#                             + (tau_h - beta + 1) ceil((l + alpha l') / n))
def _ceil(a, b):
    return -(-a // b)


def _lambda_naive_closed_form(r, l, h, lp, m, n):
    from math import gcd
    kappa = gcd(m, h)
    tau_m, tau_h = m // kappa, h // kappa
    alpha, beta = divmod(tau_m, tau_h)
    assert r % tau_m == 0, "the theorem covers whole cross-sections of lcm(m, h) rows"
    if beta == 0:
        per = tau_h * _ceil(l + (alpha - 1) * lp, n)
    else:
        per = (beta - 1) * _ceil(l + (alpha + 1) * lp, n) + (tau_h - beta + 1) * _ceil(l + alpha * lp, n)
    return (r // tau_m) * per


# (r, l, h, l', m, n): window masks (h = l' = 1, l = 2w + 1), blocked masks
# (h = l' = w, l = 2w) with m dividing h, h dividing m, and neither, and a
# few other polygons; beta = 0, beta = 1 and beta > 1 all occur
POLYGONS = [
    (24, 7, 1, 1, 4, 4),      # window w = 3, beta = 0
    (30, 9, 1, 1, 3, 5),      # window w = 4
    (32, 5, 1, 1, 16, 16),    # window w = 2, one block per patch
    (40, 17, 1, 1, 8, 3),     # window w = 8, narrow blocks
    (6, 16, 8, 8, 4, 4),      # blocked w = 8, m < h (alpha = 0, beta = 1)
    (6, 16, 8, 8, 12, 5),     # blocked, m > h, gcd 4 (alpha = 1, beta = 1)
    (10, 16, 8, 8, 20, 6),    # blocked, alpha = 2, beta = 1
    (6, 6, 3, 3, 2, 4),       # blocked w = 3, m = 2 (alpha = 0, beta = 2)
    (10, 6, 3, 3, 5, 4),      # blocked w = 3, m = 5 (alpha = 1, beta = 2)
    (15, 14, 7, 7, 3, 5),     # blocked w = 7, m = 3 (alpha = 0, beta = 3)
    (12, 7, 2, 3, 3, 4),      # h = 2, l' = 3, l = 7
    (9, 10, 4, 2, 6, 3),      # h = 4, l' = 2, l = 10
]


@pytest.mark.parametrize("r,l,h,lp,m,n", POLYGONS)
def test_naive_tiling_closed_form(r, l, h, lp, m, n):
    P = ot.structured_polygon(r, h, l, lp)
    L = max(r * h, (r - 1) * lp + l)
    anchors = ot.naive_tiling(P, L, m, n)
    assert len(anchors) == _lambda_naive_closed_form(r, l, h, lp, m, n)
    # it is an arrangement: every point is computed, anchors sit on patch rows
    met = ot.metrics(P, anchors, m, n, 1)
    assert met["blocks"] == len(anchors)
    assert all(x % m == 0 for x, _ in anchors)


def test_naive_tiling_one_block_off_fails_the_pin():
    """The closed form separates a correct count from one that is one block
    off in any patch: dropping or adding a block changes the count."""
    r, l, h, lp, m, n = POLYGONS[1]
    P = ot.structured_polygon(r, h, l, lp)
    L = max(r * h, (r - 1) * lp + l)
    want = _lambda_naive_closed_form(r, l, h, lp, m, n)
    anchors = ot.naive_tiling(P, L, m, n)
    assert len(anchors[:-1]) != want and len(anchors + [anchors[0]]) != want
    # and a patch width off by one (tiling from one column right of the
    # leftmost point) leaves points uncovered
    shifted = [(x, y + 1) for x, y in anchors]
    with pytest.raises(AssertionError):
        ot.metrics(P, shifted, m, n, 1)


def test_naive_tiling_hand_example():
    """Window w = 1 on 6 rows, m = 2, n = 2: patch rows {0,1} cover columns
    0..2 (2 blocks from column 0), {2,3} columns 1..4 (2 blocks from 1),
    {4,5} columns 3..5 (2 blocks from 3)."""
    M = om.dense_mask("window", {"w": 1}, 6)
    P = ot.points_of(M)
    assert ot.naive_tiling(P, 6, 2, 2) == [(0, 0), (0, 2), (2, 1), (2, 3), (4, 3), (4, 5)]
