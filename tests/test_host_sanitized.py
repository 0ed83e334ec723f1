"""The host planner (ACSR construction from descriptors and from masks, the
work plan, the tiling arrangements) built on its own with the address and
undefined-behaviour sanitizers (g++ -fsanitize=address,undefined), driven
through tests/native/host_check.cpp over the workload patterns, edge cases,
Hypothesis-random descriptors and masks, and compared field by field with the
regular library.  A sanitizer report ends the driver with a non-zero status,
which fails the test that sent the request.  CPU only.
"""
import json
import os
import shutil
import subprocess

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

import workloads

splat = pytest.importorskip("paper_2407_16847_amd")

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = [os.path.join(ROOT, "tests", "native", "host_check.cpp"),
       os.path.join(ROOT, "paper_2407_16847_amd", "csrc", "acsr_host.cpp"),
       os.path.join(ROOT, "paper_2407_16847_amd", "csrc", "tiling.cpp")]


@pytest.fixture(scope="module")
def driver(tmp_path_factory):
    cxx = shutil.which(os.environ.get("CXX", "g++"))
    if cxx is None:
        pytest.fail("a host C++ compiler is needed for the sanitizer build")
    exe = str(tmp_path_factory.mktemp("asan") / "host_check")
    cmd = [cxx, "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-I" + os.path.join(ROOT, "include"), *SRC, "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    return exe


def run(exe, requests):
    """Send request lines, return one parsed JSON object per line."""
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    env.pop("LD_PRELOAD", None)
    r = subprocess.run([exe], input="\n".join(requests) + "\n", capture_output=True, text=True,
                       env=env, timeout=600)
    assert r.returncode == 0, f"sanitizer run failed (exit {r.returncode}):\n{r.stderr[-4000:]}"
    assert "runtime error" not in r.stderr, r.stderr[-4000:]
    out = [json.loads(x) for x in r.stdout.splitlines()]
    assert len(out) == len(requests)
    return out


def desc_line(pattern, flags=0):
    d = pattern.desc
    vals = [d.L, flags, d.n_terms]
    for t in range(d.n_terms):
        x = d.terms[t]
        vals += [x.row_lo, x.row_hi, x.group, x.lo_i, x.lo_q, x.lo_c, x.hi_i, x.hi_q, x.hi_c, x.stride]
    return "desc " + " ".join(str(v) for v in vals)


def compare_build(got, a):
    """Driver output against the regular library's handle."""
    assert got["status"] == 0
    info = a.info()
    rp, ci = a.export()
    np.testing.assert_array_equal(np.array(got["row_ptr"]), rp)
    np.testing.assert_array_equal(np.array(got["col_idx"], dtype=np.int64), ci)
    assert (got["nnz"], got["computed"], got["n_full"], got["max_runs"]) == \
        (info["nnz"], info["computed"], info["n_full_tiles"], info["max_runs"])
    g, rows, t = a.export_plan()
    np.testing.assert_array_equal(np.array(got["groups"]).reshape(-1, 4), g.reshape(-1, 4))
    np.testing.assert_array_equal(np.array(got["rows"]), rows)
    np.testing.assert_array_equal(np.array(got["tiles"]).reshape(-1, 5), t.reshape(-1, 5))
    # one block of row masks per tile that has a PARTIAL wavefront
    assert len(got["masks"]) == 128 * int((t[:, 4] >= 0).sum()) if len(t) else True


PATTERNS = [(w.kind, w.params, w.L) for w in (workloads.get(c) for c in sorted(workloads.CONFIGS))] + [
    ("window_global", {"w": 40, "n_global": 5}, 300), ("dilated", {"w": 100, "dilation": 3}, 1000),
    ("strided_local", {"local": 50, "stride": 37}, 777), ("blocked", {"block": 64}, 130),
    ("window", {"w": 3}, 5), ("full", {}, 1), ("full", {}, 200), ("window", {"w": 700}, 513),
    ("window", {"w": 2100}, 4300), ("window", {"w": 24}, 65536)]


@pytest.mark.parametrize("kind,params,L", PATTERNS)
def test_sanitized_builds_match(driver, kind, params, L):
    pat = splat.Pattern.named(kind, params, L)
    flag_sets = [0, splat.PLAN_COLUMNS] + ([splat.PLAN_NO_SPAN] if L <= 4096 else [])
    got = run(driver, [desc_line(pat, f) for f in flag_sets])
    for f, g in zip(flag_sets, got):
        a = splat.Acsr(pat, span=not (f & splat.PLAN_NO_SPAN), columns=bool(f & splat.PLAN_COLUMNS))
        compare_build(g, a)
        if f & splat.PLAN_COLUMNS:
            assert g["columns"] == a.info()["columns"]
        a.close()


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


@settings(max_examples=150, deadline=None)
@given(affine_descs())
def test_sanitized_random_descriptors(driver, lt):
    L, terms = lt
    pat = splat.Pattern.from_terms(L, terms)
    got = run(driver, [desc_line(pat), desc_line(pat, splat.PLAN_NO_SPAN | splat.PLAN_COLUMNS)])
    try:
        a = splat.Acsr(pat)
    except splat.SplatError as e:
        assert got[0]["status"] == e.status
        return
    compare_build(got[0], a)
    b = splat.Acsr(pat, span=False, columns=True)
    compare_build(got[1], b)
    assert got[1]["columns"] == b.info()["columns"]


@settings(max_examples=60, deadline=None)
@given(st.integers(1, 40), st.integers(0, 2 ** 32 - 1), st.sampled_from([0.05, 0.3, 0.7]))
def test_sanitized_masks(driver, L, seed, p):
    """Random masks (mostly not regular) and their regular restrictions to
    one affine run per row."""
    rng = np.random.default_rng(seed)
    M = (rng.random((L, L)) < p).astype(np.uint8)
    R = np.zeros_like(M)
    for i in range(L):
        s, st_, c = int(rng.integers(0, L)), int(rng.integers(1, 5)), int(rng.integers(0, 6))
        cols = [j for j in range(s, L, st_)][:c]
        R[i, cols] = 1
    got = run(driver, ["mask %d %s" % (L, "".join(map(str, X.ravel().tolist()))) for X in (M, R)])
    for X, g in zip((M, R), got):
        try:
            a = splat.Acsr(mask=X)
        except splat.SplatError as e:
            assert g["status"] == e.status
            continue
        compare_build(g, a)


TILING = [("window", {"w": 3}, 40, 4, 4), ("blocked", {"block": 8}, 37, 4, 8),
          ("dilated", {"w": 4, "dilation": 3}, 48, 3, 3),
          ("strided_local", {"local": 5, "stride": 7}, 50, 4, 4),
          ("window_global", {"w": 3, "n_global": 2}, 33, 4, 8), ("full", {}, 20, 8, 8),
          ("window", {"w": 9}, 300, 16, 16), ("window", {"w": 40}, 1024, 32, 8)]


@pytest.mark.parametrize("kind,params,L,m,n", TILING)
def test_sanitized_tilings_match(driver, kind, params, L, m, n):
    pat = splat.Pattern.named(kind, params, L)
    reqs = [desc_line(pat)]
    calls = [("poset", 0), ("poset", 1), ("poset", 2), ("naive", 0), ("grid", 0)]
    reqs += [f"tile {splat.TILING_METHODS[meth]} {m} {n} {s}" for meth, s in calls]
    got = run(driver, reqs)
    a = splat.Acsr(pat)
    for (meth, s), g in zip(calls, got[1:]):
        want, anchors = a.tiling(meth, m, n, stretch=s, anchors=True)
        assert g["status"] == 0
        for k in ("blocks", "divergent", "redundant", "stretch", "iterations"):
            assert g[k] == want[k], (meth, s, k)
        np.testing.assert_array_equal(np.array(g["anchors"]).reshape(-1, 2), anchors.reshape(-1, 2))
