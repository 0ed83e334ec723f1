"""The checked build (libsplat_checked.so, -DSPLAT_DEBUG_BOUNDS) on the GPU.

Its kernels check every global-memory index they derive from the plan and
the ACSR runs and record any that falls outside its buffer (csrc/bounds.hpp,
splat_debug_bounds in splat.h).  Here:
  * the mechanism itself, through splat_debug_bounds_probe: an index inside
    its range comes back unchanged and records nothing; one outside comes
    back as 0 and sets exactly its kind's bit, until cleared;
  * every compute call of the C ABI, on all five workloads at full size, on
    edge cases and on random descriptor patterns: no index is ever recorded,
    and every output equals the regular library's bit for bit (the checks
    change no arithmetic).
Both libraries are driven through the C ABI directly.
"""
import ctypes

import numpy as np
import pytest
import torch

import workloads

pytestmark = pytest.mark.gpu

KINDS = {0: "row", 1: "key", 2: "value", 3: "colpos"}


@pytest.fixture(scope="module")
def libs(gpu_lib):
    splat = gpu_lib
    return splat, splat.load(), splat.load_checked()


def _flags(lib, clear=True):
    f = ctypes.c_uint32(0xFFFFFFFF)
    assert lib.splat_debug_bounds(ctypes.byref(f), 1 if clear else 0) == 0, \
        lib.splat_last_error()
    return int(f.value)


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else ctypes.c_void_p()


def _build(splat, lib, pattern, columns=False):
    h = ctypes.c_void_p()
    flags = splat.PLAN_COLUMNS if columns else 0
    rc = lib.splat_acsr_build_ex(ctypes.byref(pattern.desc), flags, ctypes.byref(h))
    assert rc == 0, lib.splat_last_error()
    info = splat.AcsrInfo()
    assert lib.splat_acsr_info(h, ctypes.byref(info)) == 0
    return h, info


def _run_all(splat, lib, pattern, w, Q, K, V):
    """Every compute call once; returns {name: output tensor}."""
    h, info = _build(splat, lib, pattern, columns=True)
    dt = 1 if w.dtype == "bf16" else 0
    B, H, d, st = w.B, w.H, w.d, _stream()
    E = B * H * int(info.nnz)
    out = {}
    try:
        for odt, name in ((0, "fused32"), (1, "fused16")):
            O = torch.empty(Q.shape, dtype=torch.float32 if odt == 0 else torch.bfloat16,
                            device="cuda")
            rc = lib.splat_sparse_mhsa_fwd(h, dt, B, H, d, _ptr(Q), _ptr(K), _ptr(V), w.scale,
                                           _ptr(O), odt, st)
            assert rc == 0, lib.splat_last_error()
            out[name] = O
        S = torch.empty(E, dtype=torch.float32, device="cuda")
        P = torch.empty(E, dtype=torch.float32, device="cuda")
        O = torch.empty(Q.shape, dtype=torch.float32, device="cuda")
        assert lib.splat_rsddmm(h, dt, B, H, d, _ptr(Q), _ptr(K), w.scale, _ptr(S), st) == 0
        assert lib.splat_row_softmax(h, B, H, _ptr(S), _ptr(P), st) == 0
        assert lib.splat_rspmm(h, dt, B, H, d, _ptr(P), _ptr(V), _ptr(O), 0, st) == 0
        out.update(S=S, P=P, unfused=O)
        if info.columns == 1:   # single-run columns: the column-major layout
            Pt = torch.empty(E, dtype=torch.float32, device="cuda")
            Oc = torch.empty(Q.shape, dtype=torch.float32, device="cuda")
            assert lib.splat_transpose_colmajor(h, B, H, _ptr(P), _ptr(Pt), st) == 0
            assert lib.splat_rspmm_colmajor(h, dt, B, H, d, _ptr(Pt), _ptr(V), _ptr(Oc), 0,
                                            st) == 0
            out.update(Pt=Pt, colmajor=Oc)
        torch.cuda.synchronize()
    finally:
        lib.splat_acsr_destroy(h)
    return out


def _compare(splat, regular, checked, pattern, w, what):
    Q, K, V = (x.cuda() for x in workloads.make_qkv(w))
    assert _flags(checked) >= 0   # cleared
    ref = _run_all(splat, regular, pattern, w, Q, K, V)
    got = _run_all(splat, checked, pattern, w, Q, K, V)
    flags = _flags(checked)
    bad = [KINDS[k] for k in KINDS if flags >> k & 1]
    assert flags == 0, f"{what}: out-of-range {bad} indices in the checked kernels"
    assert ref.keys() == got.keys()
    for name in ref:
        assert torch.equal(ref[name], got[name]), f"{what}: {name} differs from the regular build"
    return sorted(ref)


def test_probe_records_exactly_the_out_of_range_index(libs):
    _, _, chk = libs
    _flags(chk)
    r = ctypes.c_int32(-7)
    for kind in KINDS:
        assert chk.splat_debug_bounds_probe(kind, 2, 3, ctypes.byref(r)) == 0
        assert r.value == 2
        assert _flags(chk, clear=False) == 0
        for index in (3, 5, -1):
            assert chk.splat_debug_bounds_probe(kind, index, 3, ctypes.byref(r)) == 0
            assert r.value == 0
            assert _flags(chk, clear=False) == 1 << kind
        assert _flags(chk, clear=True) == 1 << kind
        assert _flags(chk) == 0


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_workloads_have_no_out_of_range_index(libs, cfg):
    splat, reg, chk = libs
    w = workloads.get(cfg)
    print(f"[gpu] checked build, workload {w.name}", flush=True)
    names = _compare(splat, reg, chk, splat.Pattern.named(w.kind, w.params, w.L), w, w.name)
    if cfg in (1, 4):   # window and dilated columns are single runs
        assert "colmajor" in names


EDGE = [("window", {"w": 0}, 1, 64), ("window", {"w": 3}, 7, 64), ("window", {"w": 40}, 130, 128),
        ("blocked", {"block": 5}, 67, 64), ("strided_local", {"local": 9, "stride": 13}, 200, 64),
        ("dilated", {"w": 20, "dilation": 3}, 257, 128),
        ("window_global", {"w": 17, "n_global": 5}, 300, 64)]


@pytest.mark.parametrize("kind,params,L,d", EDGE)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_edge_cases_have_no_out_of_range_index(libs, kind, params, L, d, dtype):
    splat, reg, chk = libs
    w = workloads.Workload(f"edge_{kind}", 2, 3, L, d, dtype, workloads.make_pattern(kind, **params),
                           1.0, 31)
    print(f"[gpu] checked build, {kind} {params} L={L} d={d} {dtype}", flush=True)
    _compare(splat, reg, chk, splat.Pattern.named(kind, params, L), w, f"{kind} L={L}")


def _term(r0, r1, lo, hi, stride=1, group=1):
    return dict(row_lo=r0, row_hi=r1, group=group, lo_i=lo[0], lo_q=lo[1], lo_c=lo[2],
                hi_i=hi[0], hi_q=hi[1], hi_c=hi[2], stride=stride)


@pytest.mark.parametrize("seed", range(8))
def test_random_patterns_have_no_out_of_range_index(libs, seed):
    """A band (stride 1 or 2) with strided causal columns and global rows
    mixed in: rows of several runs, gathered tiles, partial and empty tiles."""
    splat, reg, chk = libs
    rng = np.random.default_rng(500 + seed)
    L = int(rng.integers(30, 700))
    w1, w2 = int(rng.integers(0, L // 3)), int(rng.integers(0, L // 3))
    terms = [_term(0, L, (1, 0, -w1), (1, 0, w2), stride=int(rng.choice([1, 2])))]
    if seed % 2:
        s = int(rng.choice([5, 16]))
        terms.append(_term(int(rng.integers(0, L // 2)), L, (0, 0, int(rng.integers(0, s))),
                           (1, 0, 0), stride=s))
    if seed % 3 == 0:
        terms.append(_term(0, int(rng.integers(1, 20)), (0, 0, 0), (0, 0, L - 1)))
    try:
        pat = splat.Pattern.from_terms(L, terms)
        splat.Acsr(pat).close()
    except splat.SplatError as e:
        # a row would need more runs than the format holds: the band alone
        assert e.name == "UNSUPPORTED"
        terms = terms[:1]
        pat = splat.Pattern.from_terms(L, terms)
    d = 128 if seed % 2 else 64
    w = workloads.Workload("random", 1, 2, L, d, "bf16", ("terms", ()), 1.0, 600 + seed)
    print(f"[gpu] checked build, random seed {seed} L={L} d={d} terms={terms}", flush=True)
    _compare(splat, reg, chk, pat, w, f"random seed {seed}")
