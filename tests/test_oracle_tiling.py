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
