"""Host side of the C ABI (CPU only): symbols, ACSR construction, work plan,
the membership arithmetic and error paths, checked against the oracle's
brute-force masks.  No compute call is made here (there is no GPU).
"""
import ctypes
import os
import re
from fractions import Fraction

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

import workloads
from oracle import acsr as oacsr
from oracle import masks as om

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

splat = pytest.importorskip("paper_2407_16847_amd")


@pytest.fixture(scope="module")
def lib():
    return splat.load()


def _declared_functions():
    text = open(os.path.join(ROOT, "include", "splat.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(splat_[a-z_0-9]+)\s*\(", text)))


def test_library_exports_every_declared_symbol(lib):
    names = _declared_functions()
    assert len(names) >= 20
    for n in names:
        assert hasattr(lib, n), n
    assert lib.splat_version().startswith(b"splat-mi355x")
    checked = splat.load_checked()   # the build with device-side index checks
    for n in names:
        assert hasattr(checked, n), n


def test_index_checks_only_in_the_checked_build(lib):
    """splat_debug_bounds and its probe: unsupported in the regular build,
    argument errors caught on the host in both (no device call is made)."""
    flags, r = ctypes.c_uint32(7), ctypes.c_int32(7)
    assert lib.splat_debug_bounds(ctypes.byref(flags), 1) == 2          # UNSUPPORTED
    assert b"SPLAT_DEBUG_BOUNDS" in lib.splat_last_error()
    assert lib.splat_debug_bounds_probe(1, 5, 3, ctypes.byref(r)) == 2
    assert flags.value == 7 and r.value == 7                              # nothing written
    for l in (lib, splat.load_checked()):
        assert l.splat_debug_bounds(None, 0) == 1                         # INVALID_ARG
        assert l.splat_debug_bounds_probe(0, 0, 1, None) == 1
        assert l.splat_debug_bounds_probe(4, 0, 1, ctypes.byref(r)) == 1   # no such kind
        assert l.splat_debug_bounds_probe(-1, 0, 1, ctypes.byref(r)) == 1


def test_single_hip_runtime_in_process(lib):
    # torch is imported before libsplat: both must use one libamdhip64
    maps = open("/proc/self/maps").read()
    paths = {l.split()[-1] for l in maps.splitlines() if "libamdhip64" in l}
    assert len(paths) == 1, paths


# --------------------------------------------------------------------------
def _check_against_mask(a, M):
    L = M.shape[0]
    rp, ci = a.export()
    rp0, ci0 = om.csr(M)
    np.testing.assert_array_equal(rp, rp0)
    np.testing.assert_array_equal(ci, ci0)
    for i in range(L):
        cols = np.nonzero(M[i])[0]
        runs = a.row_runs(i)
        assert len(runs) <= splat.MAX_RUNS
        expanded = np.concatenate([np.arange(s, s + st * c, st) for s, st, c in runs]) if runs else \
            np.zeros(0, dtype=np.int64)
        np.testing.assert_array_equal(expanded, cols)
        ref = oacsr.affine_indices(cols)
        if ref is not None and len(cols) >= 1:
            # a regular row is one run; its integer (start, stride) is the paper's (a, b)
            assert len(runs) == 1
            s, stp, c = runs[0]
            assert (Fraction(1, stp), Fraction(-s, stp)) == ref and c == len(cols)
    _check_plan(a, M)


def _check_plan(a, M, span=True):
    """Every non-zero is covered by exactly one (group, tile); tile keys are in
    range and ascending; each tile holds every column of its rows inside its
    key interval; the per-wavefront states (EMPTY / PARTIAL / FULL) and the
    exported per-row tile masks equal the brute-force mask.  Without span
    specialisation (span=False) every group's tiles are the contiguous 64-key
    tiles of [0, L), and a wavefront with rows is never EMPTY."""
    L = M.shape[0]
    info = a.info()
    groups, rows, tiles = a.export_plan()
    assert sorted(rows.tolist()) == list(range(L))
    assert info["bm"] == 128 and info["bn"] == 64
    covered = np.zeros_like(M, dtype=np.int32)
    computed = 0
    prev_end = 0
    for g, (off, nrows, t0, t1) in enumerate(groups):
        assert 0 < nrows <= info["bm"] and t0 == prev_end and t1 >= t0
        prev_end = t1
        grows = rows[off:off + nrows]
        last_hi = -1
        if not span:
            starts = [tiles[t][0] for t in range(t0, t1)]
            assert starts == list(range(0, L, 64)), (g, starts[:4])
            assert all(tiles[t][1] == 1 and tiles[t][2] == min(64, L - tiles[t][0])
                       for t in range(t0, t1))
        for t in range(t0, t1):
            kb, ks, nk, flags, mblock = tiles[t]
            assert 1 <= nk <= info["bn"] and ks >= 1
            keys = kb + ks * np.arange(nk)
            assert keys[0] >= 0 and keys[-1] < L and kb > last_hi   # ascending, disjoint
            last_hi = keys[-1]
            sub = M[np.ix_(grows, keys)]
            any_partial = False
            all_full = True
            for w in range(4):
                st = (flags >> (8 + 2 * w)) & 3
                ws = sub[32 * w:32 * (w + 1)]
                if ws.shape[0] == 0 or (span and not ws.any()):
                    want = 0
                elif nk == info["bn"] and ws.all():
                    want = 3
                else:
                    want = 1
                assert st == want, (g, t, w, st, want)
                any_partial |= st == 1
                all_full &= st == 3 or ws.shape[0] == 0
                computed += 32 * 64 if st else 0
            assert bool(flags & 1) == all_full
            assert (mblock >= 0) == any_partial
            for m, i in enumerate(grows):
                bits = a.tile_row_mask(t, int(i))
                want = sum(1 << u for u in range(nk) if sub[m, u])
                assert bits == want, (g, t, i)
                inside = np.nonzero(M[i, kb:keys[-1] + 1])[0] + kb
                assert np.isin(inside, keys).all()
            covered[np.ix_(grows, keys)] += sub
    assert prev_end == len(tiles)
    assert (covered == M.astype(np.int32)).all()
    assert computed == info["computed"]
    ntiles = np.array([g[3] - g[2] for g in groups])
    assert (np.diff(ntiles) <= 0).all()                      # heaviest groups first


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_config_acsr_bit_exact(cfg):
    w = workloads.get(cfg)
    a = splat.Acsr(splat.Pattern.named(w.kind, w.params, w.L))
    M = om.dense_mask(w.kind, w.params, w.L)
    if cfg >= 4:   # full plan check is O(L^2 * rows); spot-check big configs
        rp, ci = a.export()
        rp0, ci0 = om.csr(M)
        np.testing.assert_array_equal(rp, rp0)
        np.testing.assert_array_equal(ci, ci0)
        _check_plan(a, M)
    else:
        _check_against_mask(a, M)
    info = a.info()
    assert info["nnz"] == int(M.sum()) and info["on_device"] == 0 and info["device"] == -1
    assert info["max_row_nnz"] == int(M.sum(axis=1).max())


def test_config_run_counts():
    # regular masks need one run per row; the two unions need two
    want = {1: 1, 2: 1, 3: 2, 4: 1, 5: 2}
    for cfg, n in want.items():
        w = workloads.get(cfg)
        assert splat.Acsr(splat.Pattern.named(w.kind, w.params, w.L)).info()["max_runs"] == n


def test_dilated_rows_are_regrouped_by_residue():
    # rows of one parity share their affine geometry and are planned together
    # over gathered stride-2 key tiles (section 5.2 alignment)
    w = workloads.get(4)
    a = splat.Acsr(splat.Pattern.named(w.kind, w.params, w.L))
    groups, rows, tiles = a.export_plan()
    for off, nrows, t0, t1 in groups:
        par = rows[off:off + nrows] % 2
        assert (par == par[0]).all()
        assert (tiles[t0:t1, 1] == 2).all()


# --------------------------------------------------------------------------
KINDS = st.sampled_from(["window", "blocked", "strided_local", "dilated", "window_global", "full"])


@st.composite
def named_patterns(draw):
    kind = draw(KINDS)
    L = draw(st.integers(1, 200))
    p = {}
    if kind == "window":
        p = {"w": draw(st.integers(0, 70))}
    elif kind == "blocked":
        p = {"block": draw(st.integers(1, 70))}
    elif kind == "strided_local":
        p = {"local": draw(st.integers(1, 70)), "stride": draw(st.integers(1, 70))}
    elif kind == "dilated":
        p = {"w": draw(st.integers(0, 40)), "dilation": draw(st.integers(1, 9))}
    elif kind == "window_global":
        p = {"w": draw(st.integers(0, 70)), "n_global": draw(st.integers(0, 20))}
    return kind, p, L


@settings(max_examples=120, deadline=None)
@given(named_patterns())
def test_random_named_patterns_bit_exact(pat):
    kind, p, L = pat
    a = splat.Acsr(splat.Pattern.named(kind, p, L))
    _check_against_mask(a, om.dense_mask(kind, p, L))


@st.composite
def affine_descs(draw):
    L = draw(st.integers(1, 90))
    n = draw(st.integers(0, 3))
    terms = []
    for _ in range(n):
        r0 = draw(st.integers(0, L))
        r1 = draw(st.integers(r0, L))
        terms.append(dict(row_lo=r0, row_hi=r1, group=draw(st.integers(1, 20)),
                          lo_i=draw(st.integers(-1, 1)), lo_q=draw(st.integers(-1, 1)),
                          lo_c=draw(st.integers(-40, 40)), hi_i=draw(st.integers(-1, 1)),
                          hi_q=draw(st.integers(-1, 1)), hi_c=draw(st.integers(-40, 90)),
                          stride=draw(st.sampled_from([1, 1, 2, 3, 7]))))
    return L, terms


@settings(max_examples=200, deadline=None)
@given(affine_descs())
def test_random_affine_descriptors(desc):
    L, terms = desc
    M = om.terms_mask_loops(L, terms)
    try:
        a = splat.Acsr(splat.Pattern.from_terms(L, terms))
    except splat.SplatError as e:
        # only a row needing more runs than the format holds may be refused
        assert e.name == "UNSUPPORTED" and "affine runs" in str(e)
        return
    _check_against_mask(a, M)


# --------------------------------------------------------------------------
# the paper's analysis pass on explicit masks
def test_from_mask_regular_equals_descriptor():
    for kind, p, L in [("window", {"w": 5}, 77), ("dilated", {"w": 4, "dilation": 3}, 70),
                       ("blocked", {"block": 8}, 40), ("full", {}, 33)]:
        M = om.dense_mask(kind, p, L)
        a = splat.Acsr(mask=M)
        b = splat.Acsr(splat.Pattern.named(kind, p, L))
        for x, y in zip(a.export(), b.export()):
            np.testing.assert_array_equal(x, y)
        _check_against_mask(a, M)


def test_from_mask_paper_examples():
    # P1 = {0, 2, 4, 6} in one row: a = 1/2, b = 0 -> run (0, 2, 4)
    M = np.zeros((8, 8), dtype=bool)
    M[0, [0, 2, 4, 6]] = True
    a = splat.Acsr(mask=M)
    assert a.row_runs(0) == [(0, 2, 4)]
    # P2 = {0, 2, 4, 5} is not affine-compressible: the mask is not regular
    M[0, 6] = False
    M[0, 5] = True
    with pytest.raises(splat.SplatError) as e:
        splat.Acsr(mask=M)
    assert e.value.name == "NOT_REGULAR" and "row 0" in str(e.value)


def test_from_mask_rejects_union_masks():
    for cfg in (3, 5):
        w = workloads.get(cfg)
        L = 700
        with pytest.raises(splat.SplatError) as e:
            splat.Acsr(mask=om.dense_mask(w.kind, w.params, L))
        assert e.value.name == "NOT_REGULAR"


# --------------------------------------------------------------------------
def test_error_paths(lib):
    def status(fn, *args):
        return getattr(lib, fn)(*args)

    d = splat.PatternDesc()
    h = ctypes.c_void_p()
    assert status("splat_pattern_window", 0, 3, ctypes.byref(d)) == 1
    assert status("splat_pattern_window", 10, -1, ctypes.byref(d)) == 1
    assert status("splat_pattern_blocked", 10, 0, ctypes.byref(d)) == 1
    assert status("splat_pattern_window", 10, 1, None) == 1
    assert status("splat_acsr_build", None, ctypes.byref(h)) == 1
    for bad in [dict(L=0), dict(L=70000), dict(n_terms=9), dict(stride=0), dict(group=0),
                dict(row_hi=11), dict(row_lo=5, row_hi=4), dict(lo_c=2 ** 21)]:
        d = splat.PatternDesc()
        d.L = bad.get("L", 10)
        d.n_terms = bad.get("n_terms", 1)
        t = d.terms[0]
        t.row_lo, t.row_hi = bad.get("row_lo", 0), bad.get("row_hi", 10)
        t.group, t.stride = bad.get("group", 1), bad.get("stride", 1)
        t.lo_c = bad.get("lo_c", 0)
        t.hi_c = 3
        assert status("splat_acsr_build", ctypes.byref(d), ctypes.byref(h)) == 1, bad
        assert lib.splat_last_error()
    # six runs in one row: more than SPLAT_MAX_RUNS
    terms = [dict(row_lo=0, row_hi=1, lo_c=c, hi_c=c2) for c, c2 in
             [(0, 0), (10, 11), (30, 31), (50, 51), (70, 71), (90, 90)]]
    with pytest.raises(splat.SplatError) as e:
        splat.Acsr(splat.Pattern.from_terms(100, terms))
    assert e.value.name == "UNSUPPORTED" and "row 0" in str(e.value)
    # compute on a handle built without a GPU
    a = splat.Acsr(splat.Pattern.window(64, 3))
    buf = (ctypes.c_float * 1024)()
    rc = lib.splat_sparse_mhsa_fwd(a.handle, 1, 1, 1, 64, buf, buf, buf, 0.125, buf, 1, None)
    assert rc == 6 and b"without a GPU" in lib.splat_last_error()
    rc = lib.splat_rsddmm(None, 1, 1, 1, 64, buf, buf, 0.1, buf, None)
    assert rc == 1
    # out-of-range queries
    with pytest.raises(splat.SplatError):
        a.row_runs(64)
    with pytest.raises(splat.SplatError):
        a.tile_row_mask(10 ** 6, 0)
    lib.splat_acsr_destroy(None)


def test_empty_and_tiny_masks():
    a = splat.Acsr(splat.Pattern.from_terms(5, []))
    assert a.nnz == 0 and a.export()[0].tolist() == [0] * 6
    for L in (1, 2, 3):
        a = splat.Acsr(splat.Pattern.full(L))
        _check_against_mask(a, np.ones((L, L), dtype=bool))


# --------------------------------------------------------------------------
# planning without span specialisation (the ablation of section 8.2)
@pytest.mark.parametrize("kind,params,L", [
    ("window", {"w": 4}, 300),
    ("blocked", {"block": 32}, 256),
    ("strided_local", {"local": 16, "stride": 16}, 200),
    ("dilated", {"w": 8, "dilation": 3}, 190),
    ("window_global", {"w": 20, "n_global": 5}, 260),
    ("full", {}, 70),
])
def test_no_span_plan(kind, params, L):
    pat = splat.Pattern.named(kind, params, L)
    a = splat.Acsr(pat, span=False)
    b = splat.Acsr(pat)
    M = om.dense_mask(kind, params, L)
    for x, y in zip(a.export(), b.export()):      # same index set
        np.testing.assert_array_equal(x, y)
    _check_plan(a, M, span=False)
    groups, _, _ = a.export_plan()
    n_tiles = -(-L // 64)
    want = sum(32 * 64 * n_tiles * -(-int(g[1]) // 32) for g in groups)
    assert a.info()["computed"] == want >= b.info()["computed"]


def test_no_span_plan_arguments(lib):
    d = splat.Pattern.window(100, 3).desc
    h = ctypes.c_void_p()
    assert lib.splat_acsr_build_ex(ctypes.byref(d), 4, ctypes.byref(h)) == 1
    assert b"unknown plan flags" in lib.splat_last_error()
    big = splat.Pattern.window(splat.NO_SPAN_MAX_L + 1, 3).desc
    assert lib.splat_acsr_build_ex(ctypes.byref(big), splat.PLAN_NO_SPAN, ctypes.byref(h)) == 2
    assert not h.value
    with pytest.raises(ValueError):
        splat.Acsr(mask=np.eye(8, dtype=np.uint8), span=False)
    a = splat.Acsr(splat.Pattern.window(100, 3), span=True)    # flags 0 == splat_acsr_build
    assert lib.splat_acsr_build_ex(ctypes.byref(d), 0, ctypes.byref(h)) == 0
    c = splat.Acsr.__new__(splat.Acsr)
    c._h, c._lib = h, lib
    c._info = c.info()
    assert c.info() == a.info()
    for x, y in zip(a.export_plan(), c.export_plan()):
        np.testing.assert_array_equal(x, y)


# --------------------------------------------------------------------------
# column-wise analysis and the column-major index set (section 5.2)
@pytest.mark.parametrize("kind,params,L", [
    ("window", {"w": 5}, 300), ("blocked", {"block": 16}, 250),
    ("strided_local", {"local": 9, "stride": 13}, 220), ("dilated", {"w": 7, "dilation": 3}, 200),
    ("window_global", {"w": 6, "n_global": 4}, 150), ("window_global", {"w": 200, "n_global": 4}, 150),
    ("full", {}, 70)])
def test_columns_analysis_and_csc_export(kind, params, L):
    M = om.dense_mask(kind, params, L)
    a = splat.Acsr(splat.Pattern.named(kind, params, L), columns=True)
    # the oracle's column-wise verdict: every non-empty column has affine indices
    regular = all(oacsr.affine_indices(np.nonzero(M[:, j])[0].tolist()) is not None
                  for j in range(L) if M[:, j].any())
    assert a.info()["columns"] == int(regular)
    b = splat.Acsr(splat.Pattern.named(kind, params, L))
    for x, y in zip(a.export(), b.export()):          # the row side is unchanged
        np.testing.assert_array_equal(x, y)
    if regular:
        cp, ri = a.export_csc()
        cp0, ri0 = om.csc(M)
        np.testing.assert_array_equal(cp, cp0)
        np.testing.assert_array_equal(ri, ri0)
    else:
        with pytest.raises(splat.SplatError) as e:
            a.export_csc()
        assert e.value.name == "NOT_REGULAR"


def test_columns_flag_errors(lib):
    a = splat.Acsr(splat.Pattern.window(64, 2))
    assert a.info()["columns"] == -1
    with pytest.raises(splat.SplatError) as e:
        a.export_csc()
    assert e.value.name == "INVALID_ARG"
    h = ctypes.c_void_p()
    d = splat.Pattern.window(64, 2).desc
    assert lib.splat_acsr_build_ex(ctypes.byref(d), splat.PLAN_COLUMNS | 4, ctypes.byref(h)) == 1
    both = splat.Acsr(splat.Pattern.window(100, 3), span=False, columns=True)
    assert both.info()["columns"] == 1
    _check_plan(both, om.dense_mask("window", {"w": 3}, 100), span=False)
    with pytest.raises(ValueError):
        splat.Acsr(mask=np.eye(4, dtype=np.uint8), columns=True)


# --------------------------------------------------------------------------
def _snapshot(a):
    rp, ci = a.export()
    groups, rows, tiles = a.export_plan()
    return [rp, ci, np.asarray(groups), np.asarray(rows), np.asarray(tiles)]


def test_concurrent_builds_match_serial_builds():
    """Handles built, queried and destroyed from several host threads at once
    (ctypes releases the GIL around each call) equal the same handles built
    one after the other: the build keeps no shared mutable state."""
    from concurrent.futures import ThreadPoolExecutor
    cases = [("window", {"w": 16}, 256), ("blocked", {"block": 64}, 1024),
             ("strided_local", {"local": 128, "stride": 128}, 2048),
             ("dilated", {"w": 256, "dilation": 2}, 1200),
             ("window_global", {"w": 512, "n_global": 64}, 4096),
             ("window", {"w": 3}, 5), ("full", {}, 300)]
    serial = []
    for kind, params, L in cases:
        a = splat.Acsr(splat.Pattern.named(kind, params, L))
        serial.append(_snapshot(a))
        a.close()

    def work(k):
        kind, params, L = cases[k % len(cases)]
        out = None
        for _ in range(3):
            a = splat.Acsr(splat.Pattern.named(kind, params, L))
            snap = _snapshot(a)
            a.close()
            if out is not None:
                for x, y in zip(out, snap):
                    np.testing.assert_array_equal(x, y)
            out = snap
        return k % len(cases), out

    with ThreadPoolExecutor(max_workers=8) as ex:
        for k, snap in ex.map(work, range(4 * len(cases))):
            for x, y in zip(serial[k], snap):
                np.testing.assert_array_equal(x, y)
