"""Pins for the oracle's mask enumeration and ACSR definitions (CPU only).

The mask predicates are pinned by closed-form non-zero counts (per row and in
total), by small masks written out by hand, and by the regularity structure
of each pattern; the ACSR definitions by the paper's worked examples.
"""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

import workloads
from oracle import acsr as oacsr
from oracle import masks as om

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# --------------------------------------------------------------------------
# closed-form per-row counts, written from the pattern definitions
# --------------------------------------------------------------------------
def rowcount_window(i, L, w):
    return min(i + w, L - 1) - max(i - w, 0) + 1


def rowcount_blocked(i, L, b):
    blk = i // b
    own = min(L, (blk + 1) * b) - blk * b
    prev = b if blk > 0 else 0
    return own + prev


def rowcount_strided_local(i, L, n, s):
    local = min(i, n - 1) + 1                        # [max(0, i-n+1), i]
    lo = i - n + 1                                   # strided columns strictly below lo
    below = 0 if lo <= s - 1 else (lo - 1 - (s - 1)) // s + 1
    return local + below


def rowcount_dilated(i, L, w, g):
    kmin = max(-w, -(i // g))                        # i + g*k >= 0
    kmax = min(w, (L - 1 - i) // g)                  # i + g*k <= L-1
    return kmax - kmin + 1


def rowcount_window_global(i, L, w, G):
    if i < G:
        return L
    band = rowcount_window(i, L, w)
    glob_outside = max(0, min(G, i - w))             # j < G and j < i - w
    return band + glob_outside


ROWCOUNT = {
    "window": lambda i, L, p: rowcount_window(i, L, p["w"]),
    "blocked": lambda i, L, p: rowcount_blocked(i, L, p["block"]),
    "strided_local": lambda i, L, p: rowcount_strided_local(i, L, p["local"], p["stride"]),
    "dilated": lambda i, L, p: rowcount_dilated(i, L, p["w"], p["dilation"]),
    "window_global": lambda i, L, p: rowcount_window_global(i, L, p["w"], p["n_global"]),
    "full": lambda i, L, p: L,
}

# Totals derived by hand for the five workloads.
CLOSED_FORM_NNZ = {
    1: 256 * 33 - 2 * sum(range(1, 17)),                                  # 8,176
    2: 64 * 64 + 15 * 64 * 128,                                           # 126,976
    3: sum(min(i, 127) + 1 for i in range(2048))
       + sum((i - 255) // 128 + 1 for i in range(255, 2048)),            # 267,471
    4: 3072 * 513 + 2 * (sum(i // 2 for i in range(512)) + 512 * 257),    # 1,969,664
    5: 64 * 4096 + sum(min(i + 512, 4095) - max(i - 512, 0) + 1 + max(0, min(64, i - 512))
                       for i in range(64, 4096)),                         # 4,390,336
}


def test_closed_form_totals_are_the_stated_numbers():
    assert CLOSED_FORM_NNZ == {1: 8176, 2: 126976, 3: 267471, 4: 1969664, 5: 4390336}


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_config_mask_matches_closed_forms(cfg):
    w = workloads.get(cfg)
    M = om.dense_mask(w.kind, w.params, w.L)
    counts = M.sum(axis=1)
    expect = np.array([ROWCOUNT[w.kind](i, w.L, w.params) for i in range(w.L)])
    np.testing.assert_array_equal(counts, expect)
    assert int(M.sum()) == CLOSED_FORM_NNZ[cfg]


SMALL_PATTERNS = [
    ("window", {"w": 0}), ("window", {"w": 1}), ("window", {"w": 3}), ("window", {"w": 40}),
    ("blocked", {"block": 1}), ("blocked", {"block": 3}), ("blocked", {"block": 8}),
    ("strided_local", {"local": 1, "stride": 1}), ("strided_local", {"local": 3, "stride": 4}),
    ("strided_local", {"local": 5, "stride": 2}), ("strided_local", {"local": 8, "stride": 8}),
    ("dilated", {"w": 2, "dilation": 3}), ("dilated", {"w": 5, "dilation": 2}),
    ("dilated", {"w": 1, "dilation": 1}),
    ("window_global", {"w": 2, "n_global": 3}), ("window_global", {"w": 0, "n_global": 1}),
    ("full", {}),
]


@pytest.mark.parametrize("kind,params", SMALL_PATTERNS)
@pytest.mark.parametrize("L", [1, 2, 7, 33])
def test_small_masks_vectorised_equals_loops_and_row_counts(kind, params, L):
    M = om.dense_mask(kind, params, L)
    np.testing.assert_array_equal(M, om.dense_mask_loops(kind, params, L))
    counts = [ROWCOUNT[kind](i, L, params) for i in range(L)]
    np.testing.assert_array_equal(M.sum(axis=1), counts)
    for i in range(L):
        np.testing.assert_array_equal(om.row_columns(kind, params, L, i), np.nonzero(M[i])[0])


def _from_rows(L, rows):
    M = np.zeros((L, L), dtype=bool)
    for i, cols in enumerate(rows):
        M[i, cols] = True
    return M


def test_hand_written_small_masks():
    # window w=1, L=4: tridiagonal
    assert (om.dense_mask("window", {"w": 1}, 4) ==
            _from_rows(4, [[0, 1], [0, 1, 2], [1, 2, 3], [2, 3]])).all()
    # blocked, block 2, L=6: own block and previous block
    assert (om.dense_mask("blocked", {"block": 2}, 6) ==
            _from_rows(6, [[0, 1], [0, 1], [0, 1, 2, 3], [0, 1, 2, 3], [2, 3, 4, 5], [2, 3, 4, 5]])).all()
    # strided + local, local 2, stride 3, L=7: j in [i-1, i] or (j % 3 == 2 and j <= i)
    assert (om.dense_mask("strided_local", {"local": 2, "stride": 3}, 7) ==
            _from_rows(7, [[0], [0, 1], [1, 2], [2, 3], [2, 3, 4], [2, 4, 5], [2, 5, 6]])).all()
    # dilated, dilation 2, w 1, L=6: j in {i-2, i, i+2}
    assert (om.dense_mask("dilated", {"w": 1, "dilation": 2}, 6) ==
            _from_rows(6, [[0, 2], [1, 3], [0, 2, 4], [1, 3, 5], [2, 4], [3, 5]])).all()
    # window + global, w 1, 1 global token, L=5
    assert (om.dense_mask("window_global", {"w": 1, "n_global": 1}, 5) ==
            _from_rows(5, [[0, 1, 2, 3, 4], [0, 1, 2], [0, 1, 2, 3], [0, 2, 3, 4], [0, 3, 4]])).all()


def test_structure_of_the_five_masks():
    m1 = om.dense_mask("window", {"w": 16}, 256)
    assert (m1 == m1.T).all()                                   # symmetric band
    m3 = om.dense_mask("strided_local", {"local": 128, "stride": 128}, 2048)
    assert not np.triu(m3, 1).any()                             # causal
    assert m3[:, 127::128].sum() == sum(2048 - j for j in range(127, 2048, 128))
    m4 = om.dense_mask("dilated", {"w": 256, "dilation": 2}, 4096)
    ii, jj = np.nonzero(m4)
    assert ((ii - jj) % 2 == 0).all()                           # parity preserved
    m5 = om.dense_mask("window_global", {"w": 512, "n_global": 64}, 4096)
    assert m5[:64].all() and m5[:, :64].all()                   # global rows and columns


def test_csr_order_is_row_major_ascending():
    M = om.dense_mask("strided_local", {"local": 3, "stride": 4}, 13)
    row_ptr, col = om.csr(M)
    assert row_ptr[0] == 0 and row_ptr[-1] == M.sum()
    for i in range(13):
        seg = col[row_ptr[i]:row_ptr[i + 1]]
        assert (np.diff(seg) > 0).all()
        np.testing.assert_array_equal(seg, np.nonzero(M[i])[0])


# --------------------------------------------------------------------------
# ACSR definitions
# --------------------------------------------------------------------------
def _golden():
    with open(os.path.join(GOLDEN, "paper_examples.json")) as f:
        return json.load(f)


def test_paper_example_affine_compressibility():
    for ex in _golden()["affine_compressible"]:
        pts = [tuple(p) for p in ex["points"]]
        assert oacsr.is_affine_compressible(pts) == ex["compressible"]
        if ex["compressible"]:
            a, b = oacsr.affine_indices([x for x, _ in pts])
            assert a == Fraction(ex["a"]) and b == Fraction(ex["b"])


def test_paper_example_dense_column():
    for ex in _golden()["dense_column"]:
        a, b = Fraction(ex["a"]), Fraction(ex["b"])
        assert oacsr.dense_col(ex["sparse_i"], a, b) == ex["dense_col"]
        # the row is columns b'..: sparse positions 0..nnzs-1 map to 1, 2, 3, 4
        cols = [int(oacsr.dense_col(s, a, b)) for s in range(ex["nnzs"])]
        assert cols == [1, 2, 3, 4]
        assert oacsr.affine_indices(cols) == (a, b)


def test_solve_on_arithmetic_progressions():
    for start in (0, 3, 17):
        for stride in (1, 2, 5, 128):
            cols = [start + stride * t for t in range(6)]
            a, b = oacsr.affine_indices(cols)
            assert a == Fraction(1, stride) and b == Fraction(-start, stride)
            assert [oacsr.sparse_index(c, a, b) for c in cols] == list(range(6))
            assert [oacsr.dense_col(s, a, b) for s in range(6)] == cols
    assert oacsr.affine_indices([0, 2, 4, 5]) is None
    assert oacsr.affine_indices([7]) == (1, -7)
    assert oacsr.affine_indices([]) == (1, 0)


def test_fast_indexing_membership_matches_mask_on_regular_rows():
    for kind, params, L in [("window", {"w": 3}, 20), ("dilated", {"w": 3, "dilation": 3}, 25),
                            ("blocked", {"block": 4}, 16)]:
        M = om.dense_mask(kind, params, L)
        for i in range(L):
            cols = np.nonzero(M[i])[0]
            a, b = oacsr.affine_indices(cols)
            for j in range(L):
                assert oacsr.contains(j, a, b, len(cols)) == bool(M[i, j])


@pytest.mark.parametrize("cfg,n_irregular", [(1, 0), (2, 0), (3, 1792), (4, 0), (5, 3519)])
def test_regularity_of_the_five_masks(cfg, n_irregular):
    # cfg 3: rows 256.. carry a strided column detached from the local window
    # (row 255's column 127 abuts its window 128..255); cfg 5: rows 577.. have
    # the global columns 0..63 detached from the band [i-512, i+512].
    w = workloads.get(cfg)
    M = om.dense_mask(w.kind, w.params, w.L)
    bad = sum(oacsr.affine_indices(np.nonzero(r)[0]) is None for r in M)
    assert bad == n_irregular
    assert oacsr.is_regular(M) == (n_irregular == 0)


@pytest.mark.parametrize("kind,params", SMALL_PATTERNS)
def test_row_masks_equal_dense_mask(kind, params):
    L = 29
    M = om.dense_mask(kind, params, L)
    rows = om.row_columns_fast(kind, params, L, range(L))
    for i in range(L):
        np.testing.assert_array_equal(rows[i], np.nonzero(M[i])[0])


# --------------------------------------------------------------------------
# masks from affine-term descriptors
def _term(row_lo, row_hi, lo, hi, stride=1, group=1):
    """lo, hi: (coefficient of i, coefficient of q, constant)."""
    return dict(row_lo=row_lo, row_hi=row_hi, group=group, lo_i=lo[0], lo_q=lo[1], lo_c=lo[2],
                hi_i=hi[0], hi_q=hi[1], hi_c=hi[2], stride=stride)


def test_terms_mask_matches_named_patterns():
    """Hand-written term lists for the named patterns give their predicates' masks."""
    L = 97
    cases = [
        (("window", {"w": 5}), [_term(0, L, (1, 0, -5), (1, 0, 5))]),
        (("dilated", {"w": 4, "dilation": 3}), [_term(0, L, (1, 0, -12), (1, 0, 12), stride=3)]),
        (("blocked", {"block": 8}), [_term(0, L, (0, 1, -8), (0, 1, 7), group=8)]),
        (("window_global", {"w": 6, "n_global": 4}),
         [_term(0, L, (1, 0, -6), (1, 0, 6)), _term(0, 4, (0, 0, 0), (0, 0, L - 1)),
          _term(0, L, (0, 0, 0), (0, 0, 3))]),
        (("strided_local", {"local": 10, "stride": 7}),
         [_term(0, L, (1, 0, -9), (1, 0, 0)), _term(0, L, (0, 0, 6), (1, 0, 0), stride=7)]),
        (("full", {}), [_term(0, L, (0, 0, 0), (0, 0, L - 1))]),
    ]
    for (kind, params), terms in cases:
        ref = om.dense_mask(kind, params, L)
        np.testing.assert_array_equal(om.terms_mask(L, terms), ref, err_msg=kind)
        np.testing.assert_array_equal(om.terms_mask_loops(L, terms), ref, err_msg=kind)


def test_terms_mask_grid_equals_loops_on_random_terms():
    rng = np.random.default_rng(11)
    for _ in range(60):
        L = int(rng.integers(1, 60))
        terms = []
        for _ in range(int(rng.integers(0, 4))):
            r0 = int(rng.integers(0, L + 1))
            r1 = int(rng.integers(r0, L + 1))
            terms.append(_term(r0, r1, (int(rng.integers(-1, 2)), int(rng.integers(-1, 2)),
                                        int(rng.integers(-30, 30))),
                               (int(rng.integers(-1, 2)), int(rng.integers(-1, 2)),
                                int(rng.integers(-30, 70))),
                               stride=int(rng.choice([1, 2, 3, 7])), group=int(rng.integers(1, 12))))
        np.testing.assert_array_equal(om.terms_mask(L, terms), om.terms_mask_loops(L, terms))


def test_terms_mask_clamping_keeps_the_residue():
    """Columns below 0 are dropped, not shifted: a stride-3 term starting at -4
    keeps only columns congruent to -4 (mod 3), i.e. 2, 5, 8, ..."""
    M = om.terms_mask(12, [_term(0, 1, (0, 0, -4), (0, 0, 11), stride=3)])
    assert np.flatnonzero(M[0]).tolist() == [2, 5, 8, 11]


# --------------------------------------------------------------------------
# column-compressed, column-major order (section 5.2)
def test_csc_hand_worked_example():
    import json
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "colmajor_example.json")))
    M = np.array(g["mask"], dtype=bool)
    rp, ci = om.csr(M)
    cp, ri = om.csc(M)
    assert rp.tolist() == g["row_ptr"] and ci.tolist() == g["col_idx"]
    assert cp.tolist() == g["col_ptr"] and ri.tolist() == g["row_idx"]
    assert om.colmajor_source(M).tolist() == g["colmajor_source"]


@pytest.mark.parametrize("kind,params,L", [
    ("window", {"w": 3}, 40), ("blocked", {"block": 8}, 37), ("strided_local", {"local": 5, "stride": 7}, 50),
    ("dilated", {"w": 4, "dilation": 3}, 45), ("window_global", {"w": 2, "n_global": 3}, 30)])
def test_csc_properties(kind, params, L):
    M = om.dense_mask(kind, params, L)
    rp, ci = om.csr(M)
    cp, ri = om.csc(M)
    src = om.colmajor_source(M)
    assert (np.diff(cp) == M.sum(axis=0)).all()
    for j in range(L):
        rows = ri[cp[j]:cp[j + 1]]
        np.testing.assert_array_equal(rows, np.nonzero(M[:, j])[0])     # the column, ascending
        for t, i in enumerate(rows):
            k = src[cp[j] + t]                                          # its CSR slot
            assert rp[i] <= k < rp[i + 1] and ci[k] == j
    assert sorted(src.tolist()) == list(range(int(M.sum())))            # a permutation
    # going through the transpose and back is the identity
    back = om.colmajor_source(M.T)
    np.testing.assert_array_equal(src[back], np.arange(int(M.sum())))
