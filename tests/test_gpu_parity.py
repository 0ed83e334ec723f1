"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle.

Tolerances (stated by the target and derived in the comments):
  * bf16 inputs: elementwise |O - O_ref| <= 2e-2 (O_ref is fp64 on the same
    bf16-rounded inputs);
  * fp32 inputs: per-row normwise max_i ||O_i - R_i||_inf / ||R_i||_inf <= 1e-5;
  * unfused intermediates: each score S_ij within 1e-5 of the magnitude of
    its terms, |S_ij - R_ij| <= 1e-5 * scale * sum_c |q_ic k_jc| (the forward
    error of a d-term fp32 dot product is at most about d * 2^-24 of that
    magnitude: 3.8e-6 at d = 64, 7.6e-6 at d = 128; a score near 0 after
    cancellation has no small relative error, so the bound is not taken
    relative to |R_ij| or to its row);
    P elementwise <= 1e-5 (S error times P plus fp32 exp/divide rounding),
    every row of P sums to 1 within 1e-5.
Sizes: every workload at full size against the dense oracle, the two
L = 4096 workloads in the launch the benchmark times: every row of every head
of O, and S and P on four whole heads.
"""
import math

import numpy as np
import pytest
import torch

import workloads
from oracle import attention as oa
from oracle import masks as om

pytestmark = pytest.mark.gpu

BF16_ABS = 2e-2
F32_REL = 1e-5
S_REL = 1e-5
P_ABS = 1e-5


def _dev(t):
    return t.to("cuda")


def _rows_normwise(x, ref):
    """max over rows of ||x_i - r_i||_inf / ||r_i||_inf, rows of the last axis."""
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    num = np.abs(x - ref).max(axis=-1)
    den = np.abs(ref).max(axis=-1)
    zero = den == 0
    assert (num[zero] == 0).all(), "rows whose reference is 0 must be exactly 0"
    return float((num[~zero] / den[~zero]).max()) if (~zero).any() else 0.0


def check_O(O, ref, dtype, what=""):
    O = O.float().cpu().numpy().astype(np.float64)
    assert np.isfinite(O).all(), f"{what}: non-finite output"
    if dtype == "bf16":
        err = float(np.abs(O - ref).max())
        assert err <= BF16_ABS, f"{what}: max abs error {err:.3e} > {BF16_ABS}"
    else:
        err = _rows_normwise(O, ref)
        assert err <= F32_REL, f"{what}: row-normwise rel error {err:.3e} > {F32_REL}"
    return err


def unfused(a, splat, Q, K, V, scale, out_dtype):
    S = splat.rsddmm(a, Q, K, scale)
    P = splat.row_softmax(a, S)
    O = splat.rspmm(a, P, V, out_dtype=out_dtype)
    return S, P, O


def _score_err(s, ref, qi, k_cols, scale):
    """max |s - ref| / (scale * sum_c |q_ic k_jc|) over one row's scores."""
    mag = scale * (np.abs(k_cols) @ np.abs(qi))
    err = np.abs(np.asarray(s, dtype=np.float64) - ref)
    zero = mag == 0
    assert (err[zero] == 0).all(), "scores whose terms are all 0 must be exactly 0"
    return float((err[~zero] / mag[~zero]).max()) if (~zero).any() else 0.0


def _s_err_csr(x, ref, q, k, row_ptr, col_idx, scale):
    """_score_err over every row of one head (CSR arrays, q and k fp64 [L, d])."""
    worst = 0.0
    for i in range(len(row_ptr) - 1):
        lo, hi = row_ptr[i], row_ptr[i + 1]
        if hi > lo:
            worst = max(worst, _score_err(x[lo:hi], ref[lo:hi], q[i], k[col_idx[lo:hi]], scale))
    return worst


# --------------------------------------------------------------------------
@pytest.mark.parametrize("cfg", [1, 2, 3])
def test_small_configs_full_oracle(gpu_lib, record_errors, cfg):
    splat = gpu_lib
    w = workloads.get(cfg)
    print(f"[gpu] cfg{cfg} {w.name} full-size dense oracle", flush=True)
    Q, K, V = workloads.make_qkv(w)
    M = om.dense_mask(w.kind, w.params, w.L)
    ref, Sref, Pref = oa.masked_attention(Q, K, V, M, w.scale, want_csr=True)
    a = splat.Acsr(splat.Pattern.named(w.kind, w.params, w.L))
    Qd, Kd, Vd = _dev(Q), _dev(K), _dev(V)
    errs = {}
    for odt in (torch.float32, torch.bfloat16):
        O = splat.sparse_mhsa_fwd(a, Qd, Kd, Vd, w.scale, out_dtype=odt)
        torch.cuda.synchronize()
        errs[f"fused/{odt}"] = check_O(O, ref, w.dtype if odt == torch.float32 else "bf16",
                                       f"cfg{cfg} fused out={odt}")
    S, P, O = unfused(a, splat, Qd, Kd, Vd, w.scale, torch.float32)
    O16 = splat.rspmm(a, P, Vd, out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    errs["unfused"] = check_O(O, ref, w.dtype, f"cfg{cfg} unfused")
    errs["unfused/bf16"] = check_O(O16, ref, "bf16", f"cfg{cfg} unfused out=bf16")
    S, P = S.cpu().numpy(), P.cpu().numpy()
    rp, ci = om.csr(M)
    q, k = oa.to_f64(Q), oa.to_f64(K)
    for b in range(w.B):
        for h in range(w.H):
            np.testing.assert_array_less(np.abs(P[b, h] - Pref[b, h]), P_ABS)
            err = _s_err_csr(S[b, h], Sref[b, h], q[b, h], k[b, h], rp, ci, w.scale)
            assert err <= S_REL, f"S rel {err}"
    print(f"[gpu] cfg{cfg} errors {errs}", flush=True)
    record_errors(f"cfg{cfg} {w.name}", errs)


def _sample_rows(L, extra, rng, n_random=40):
    rows = set(r for r in extra if 0 <= r < L)
    rows.update(rng.integers(0, L, size=n_random).tolist())
    return sorted(rows)


def _s_err_dense(s_csr, ref_csr, q, k, mask, scale):
    """_score_err over every score of one head at once: the magnitude
    scale * sum_c |q_ic k_jc| is one dense product of |q| and |k|^T,
    gathered at the mask in CSR order."""
    mag = (scale * (np.abs(q) @ np.abs(k).T))[mask]
    err = np.abs(np.asarray(s_csr, dtype=np.float64) - ref_csr)
    zero = mag == 0
    assert (err[zero] == 0).all(), "scores whose terms are all 0 must be exactly 0"
    return float((err[~zero] / mag[~zero]).max()) if (~zero).any() else 0.0


@pytest.mark.parametrize("cfg", [4, 5])
def test_large_configs_every_row(gpu_lib, record_errors, cfg):
    """Full size, the benchmark's launch (bf16 in; fp32 and bf16 out): every
    row of every head of the fused and the unfused output against the dense
    fp64 oracle, and S and P element by element on four whole heads."""
    splat = gpu_lib
    w = workloads.get(cfg)
    print(f"[gpu] cfg{cfg} {w.name} full size, every row of every head", flush=True)
    Q, K, V = workloads.make_qkv(w)
    a = splat.Acsr(splat.Pattern.named(w.kind, w.params, w.L))
    Qd, Kd, Vd = _dev(Q), _dev(K), _dev(V)
    O32 = splat.sparse_mhsa_fwd(a, Qd, Kd, Vd, w.scale, out_dtype=torch.float32)
    O16 = splat.sparse_mhsa_fwd(a, Qd, Kd, Vd, w.scale, out_dtype=torch.bfloat16)
    S, P, Ou = unfused(a, splat, Qd, Kd, Vd, w.scale, torch.float32)
    torch.cuda.synchronize()
    outs = {"fused32": O32.cpu().numpy(), "fused16": O16.float().cpu().numpy(),
            "unfused": Ou.cpu().numpy()}
    del O32, O16, Ou
    M = om.dense_mask(w.kind, w.params, w.L)
    q, k, v = oa.to_f64(Q), oa.to_f64(K), oa.to_f64(V)
    heads = [(0, 0), (0, w.H - 1), (w.B - 1, w.H // 2), (w.B - 1, w.H - 1)]
    rp, _ = a.export()
    worst = {name: 0.0 for name in outs}
    worst.update(S=0.0, P=0.0, rowsum=0.0)
    for b in range(w.B):
        for h in range(w.H):
            Sd, Pd, Or = oa.attention_head(q[b, h], k[b, h], v[b, h], M, w.scale)
            for name, O in outs.items():
                assert np.isfinite(O[b, h]).all(), f"cfg{cfg} {name} head {(b, h)}: non-finite"
                err = float(np.abs(O[b, h].astype(np.float64) - Or).max())
                worst[name] = max(worst[name], err)
                assert err <= BF16_ABS, f"cfg{cfg} {name} head {(b, h)}: {err:.3e}"
            if (b, h) in heads:
                Sg = S[b, h].cpu().numpy()
                Pg = P[b, h].cpu().numpy().astype(np.float64)
                es = _s_err_dense(Sg, Sd[M], q[b, h], k[b, h], M, w.scale)
                ep = float(np.abs(Pg - Pd[M]).max())
                sums = np.add.reduceat(Pg, rp[:-1][np.diff(rp) > 0])
                er = float(np.abs(sums - 1.0).max())
                worst["S"], worst["P"] = max(worst["S"], es), max(worst["P"], ep)
                worst["rowsum"] = max(worst["rowsum"], er)
                assert es <= S_REL, f"cfg{cfg} head {(b, h)}: S rel error {es:.3e}"
                assert ep <= P_ABS, f"cfg{cfg} head {(b, h)}: P abs error {ep:.3e}"
                assert er <= 1e-5, f"cfg{cfg} head {(b, h)}: P row sum off by {er:.3e}"
            del Sd, Pd
    print(f"[gpu] cfg{cfg} max errors over all {w.B * w.H} heads: "
          + ", ".join(f"{k} {v:.3e}" for k, v in worst.items()), flush=True)
    record_errors(f"cfg{cfg} {w.name} (all {w.B * w.H} heads)", worst)


# --------------------------------------------------------------------------
# edge cases: ragged sizes, d = 128, tiny L, empty rows, full and diagonal masks
EDGE = [
    ("window_global", {"w": 40, "n_global": 5}, 300, 64),
    ("dilated", {"w": 100, "dilation": 3}, 1000, 128),
    ("strided_local", {"local": 50, "stride": 37}, 777, 64),
    ("blocked", {"block": 64}, 130, 128),
    ("window", {"w": 3}, 5, 64),
    ("full", {}, 1, 64),
    ("full", {}, 200, 64),
    ("window", {"w": 700}, 513, 128),
    # rows longer than 4096 values: the softmax takes its streaming path
    ("window", {"w": 2100}, 4300, 64),
]


@pytest.mark.parametrize("kind,params,L,d", EDGE)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_edge_cases(gpu_lib, kind, params, L, d, dtype):
    splat = gpu_lib
    w = workloads.Workload("edge", 2, 3, L, d, dtype, workloads.make_pattern(kind, **params), 1.0, L + d)
    print(f"[gpu] edge {kind} {params} L={L} d={d} {dtype}", flush=True)
    Q, K, V = workloads.make_qkv(w)
    M = om.dense_mask(kind, params, L)
    ref, Sref, Pref = oa.masked_attention(Q, K, V, M, w.scale, want_csr=True)
    a = splat.Acsr(splat.Pattern.named(kind, params, L))
    Qd, Kd, Vd = _dev(Q), _dev(K), _dev(V)
    O = splat.sparse_mhsa_fwd(a, Qd, Kd, Vd, w.scale, out_dtype=torch.float32)
    S, P, Ou = unfused(a, splat, Qd, Kd, Vd, w.scale, torch.float32)
    torch.cuda.synchronize()
    check_O(O, ref, dtype, "fused")
    check_O(Ou, ref, dtype, "unfused")
    S, P = S.cpu().numpy(), P.cpu().numpy()
    rp, ci = om.csr(M)
    q, k = oa.to_f64(Q), oa.to_f64(K)
    for b in range(2):
        for h in range(3):
            assert _s_err_csr(S[b, h], Sref[b, h], q[b, h], k[b, h], rp, ci, w.scale) <= S_REL
            assert np.abs(P[b, h] - Pref[b, h]).max() <= P_ABS


# plans without span specialisation (every group walks all of [0, L), with
# tiles in which some wavefronts have no key at all): same results
NO_SPAN = [
    ("window", {"w": 8}, 1024, 64),
    ("blocked", {"block": 64}, 1024, 64),
    ("strided_local", {"local": 32, "stride": 32}, 1000, 64),
    ("dilated", {"w": 40, "dilation": 3}, 700, 128),
    ("window_global", {"w": 20, "n_global": 7}, 333, 64),
]


@pytest.mark.parametrize("kind,params,L,d", NO_SPAN)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_no_span_plans(gpu_lib, kind, params, L, d, dtype):
    splat = gpu_lib
    w = workloads.Workload("nospan", 2, 3, L, d, dtype, workloads.make_pattern(kind, **params), 1.0,
                           L + 3 * d)
    print(f"[gpu] no-span {kind} {params} L={L} d={d} {dtype}", flush=True)
    Q, K, V = workloads.make_qkv(w)
    M = om.dense_mask(kind, params, L)
    ref, Sref, Pref = oa.masked_attention(Q, K, V, M, w.scale, want_csr=True)
    a = splat.Acsr(splat.Pattern.named(kind, params, L), span=False)
    Qd, Kd, Vd = _dev(Q), _dev(K), _dev(V)
    O = splat.sparse_mhsa_fwd(a, Qd, Kd, Vd, w.scale, out_dtype=torch.float32)
    Ob = splat.sparse_mhsa_fwd(a, Qd, Kd, Vd, w.scale)
    S, P, Ou = unfused(a, splat, Qd, Kd, Vd, w.scale, torch.float32)
    torch.cuda.synchronize()
    check_O(O, ref, dtype, "fused")
    check_O(Ob, ref, dtype, "fused, input-dtype output")
    check_O(Ou, ref, dtype, "unfused")
    S, P = S.cpu().numpy(), P.cpu().numpy()
    rp, ci = om.csr(M)
    q, k = oa.to_f64(Q), oa.to_f64(K)
    for b in range(2):
        for h in range(3):
            assert _s_err_csr(S[b, h], Sref[b, h], q[b, h], k[b, h], rp, ci, w.scale) <= S_REL
            assert np.abs(P[b, h] - Pref[b, h]).max() <= P_ABS


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_diagonal_mask_returns_v_exactly(gpu_lib, dtype):
    splat = gpu_lib
    w = workloads.Workload("diag", 2, 2, 333, 64, dtype, workloads.make_pattern("window", w=0), 1.0, 7)
    Q, K, V = (_dev(x) for x in workloads.make_qkv(w))
    a = splat.Acsr(splat.Pattern.window(w.L, 0))
    odt = torch.float32 if dtype == "f32" else torch.bfloat16
    O = splat.sparse_mhsa_fwd(a, Q, K, V, w.scale, out_dtype=odt)
    Ou = splat.rspmm(a, splat.row_softmax(a, splat.rsddmm(a, Q, K, w.scale)), V, out_dtype=odt)
    torch.cuda.synchronize()
    assert torch.equal(O, V) and torch.equal(Ou, V)


def test_empty_rows_give_zero(gpu_lib):
    splat = gpu_lib
    L = 260
    # rows [0, 100) and [200, 260) attend to a window; rows [100, 200) to nothing
    terms = [dict(row_lo=0, row_hi=100, lo_i=1, lo_c=-5, hi_i=1, hi_c=5),
             dict(row_lo=200, row_hi=L, lo_i=1, lo_c=-70, hi_i=1, hi_c=0)]
    a = splat.Acsr(splat.Pattern.from_terms(L, terms))
    M = np.zeros((L, L), dtype=bool)
    for i in range(L):
        if i < 100:
            M[i, max(0, i - 5):min(L, i + 6)] = True
        elif i >= 200:
            M[i, i - 70:i + 1] = True
    assert a.nnz == int(M.sum())
    for dtype in ("f32", "bf16"):
        w = workloads.Workload("empty", 1, 2, L, 128, dtype, workloads.make_pattern("full"), 1.0, 3)
        Q, K, V = workloads.make_qkv(w)
        ref = oa.masked_attention(Q, K, V, M, w.scale)
        Qd, Kd, Vd = _dev(Q), _dev(K), _dev(V)
        O = splat.sparse_mhsa_fwd(a, Qd, Kd, Vd, w.scale, out_dtype=torch.float32)
        Ou = splat.rspmm(a, splat.row_softmax(a, splat.rsddmm(a, Qd, Kd, w.scale)), Vd,
                         out_dtype=torch.float32)
        torch.cuda.synchronize()
        assert (O[:, :, 100:200] == 0).all() and (Ou[:, :, 100:200] == 0).all()
        check_O(O, ref, dtype, "fused empty rows")
        check_O(Ou, ref, dtype, "unfused empty rows")


def test_softmax_in_place_and_determinism(gpu_lib):
    splat = gpu_lib
    w = workloads.get(2)
    Q, K, V = (_dev(x) for x in workloads.make_qkv(w))
    a = splat.Acsr(splat.Pattern.named(w.kind, w.params, w.L))
    S = splat.rsddmm(a, Q, K, w.scale)
    P = splat.row_softmax(a, S)
    S2 = S.clone()
    P2 = splat.row_softmax(a, S2, S2)       # in place
    O1 = splat.sparse_mhsa_fwd(a, Q, K, V, w.scale)
    O2 = splat.sparse_mhsa_fwd(a, Q, K, V, w.scale)
    torch.cuda.synchronize()
    assert P2.data_ptr() == S2.data_ptr() and torch.equal(P, P2)
    assert torch.equal(O1, O2)


def test_argument_errors(gpu_lib):
    splat = gpu_lib
    a = splat.Acsr(splat.Pattern.window(128, 4))
    x = torch.zeros((1, 1, 128, 64), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(ValueError):
        splat.sparse_mhsa_fwd(a, torch.zeros((1, 1, 64, 64), dtype=torch.bfloat16, device="cuda"), x, x, 0.1)
    with pytest.raises(splat.SplatError) as e:
        splat.sparse_mhsa_fwd(a, torch.zeros((1, 1, 128, 32), dtype=torch.bfloat16, device="cuda"),
                              torch.zeros((1, 1, 128, 32), dtype=torch.bfloat16, device="cuda"),
                              torch.zeros((1, 1, 128, 32), dtype=torch.bfloat16, device="cuda"), 0.1)
    assert e.value.name == "UNSUPPORTED"
    lib = splat.load()
    rc = lib.splat_sparse_mhsa_fwd(a.handle, 1, 1, 1, 64, x.data_ptr() + 2, x.data_ptr(), x.data_ptr(),
                                   0.1, x.data_ptr(), 1, None)
    assert rc == 1 and b"aligned" in lib.splat_last_error()
    info = a.info()
    assert info["on_device"] == 1 and info["device"] == torch.cuda.current_device()


def test_binding_rejects_mismatched_tensors(gpu_lib):
    """The binding checks every caller-supplied output and workspace against
    Q/V's shape and device before anything is launched: an O of the wrong
    batch or head count would otherwise be written past its end, and a host
    tensor's pointer would reach a kernel."""
    splat = gpu_lib
    L, d = 128, 64
    a = splat.Acsr(splat.Pattern.window(L, 4))
    B, H = 2, 3
    x = torch.randn((B, H, L, d), device="cuda").to(torch.bfloat16)
    small = torch.zeros((1, 1, L, d), dtype=torch.float32, device="cuda")
    S = splat.rsddmm(a, x, x, 0.1)
    P = splat.row_softmax(a, S)
    torch.cuda.synchronize()
    before = small.clone()
    with pytest.raises(ValueError):
        splat.sparse_mhsa_fwd(a, x, x, x, 0.1, O=small)
    with pytest.raises(ValueError):
        splat.rspmm(a, P, x, O=small)
    with pytest.raises(ValueError):
        splat.sparse_mhsa_unfused(a, x, x, x, 0.1, O=small)
    with pytest.raises(ValueError):
        splat.rsddmm(a, x, x, 0.1, S=torch.empty((1, 1, a.nnz), device="cuda"))
    with pytest.raises(ValueError):
        splat.row_softmax(a, S, P=torch.empty((1, H, a.nnz), device="cuda"))
    with pytest.raises(TypeError):
        splat.rsddmm(a, x, x, 0.1, S=torch.empty((B, H, a.nnz)))
    with pytest.raises(TypeError):
        splat.row_softmax(a, S.cpu())
    with pytest.raises(TypeError):
        splat.row_softmax(a, S, P=torch.empty((B, H, a.nnz)))
    with pytest.raises(TypeError):
        splat.rspmm(a, P.cpu(), x)
    with pytest.raises(TypeError):
        splat.sparse_mhsa_fwd(a, x, x, x.cpu(), 0.1)
    torch.cuda.synchronize()
    assert torch.equal(small, before), "a rejected call wrote its output"


# --------------------------------------------------------------------------
# random affine-term descriptors: rows with several runs, strided (gathered)
# tiles, partial tiles and empty rows, through the fused and unfused paths
def _random_terms(rng, L):
    """A band over all rows (stride 1 or 2) plus some of: strided causal
    columns, a blocked term, global rows -- rows then mix several runs."""
    def term(r0, r1, lo, hi, stride=1, group=1):
        return dict(row_lo=r0, row_hi=r1, group=group, lo_i=lo[0], lo_q=lo[1], lo_c=lo[2],
                    hi_i=hi[0], hi_q=hi[1], hi_c=hi[2], stride=stride)
    w1, w2 = int(rng.integers(0, L // 3)), int(rng.integers(0, L // 3))
    terms = [term(0, L, (1, 0, -w1), (1, 0, w2), stride=int(rng.choice([1, 2])))]
    if rng.random() < 0.6:
        r0 = int(rng.integers(0, L // 2))
        s = int(rng.choice([3, 5, 16]))
        terms.append(term(r0, L, (0, 0, int(rng.integers(0, s))), (1, 0, 0), stride=s))
    if rng.random() < 0.4:
        g = int(rng.choice([8, 32, 64]))
        terms.append(term(0, L, (0, 1, -g), (0, 1, g - 1), group=g))
    if rng.random() < 0.4:
        terms.append(term(0, int(rng.integers(1, 40)), (0, 0, 0), (0, 0, L - 1)))
    return terms


@pytest.mark.parametrize("seed", range(12))
def test_random_descriptor_patterns(gpu_lib, seed):
    splat = gpu_lib
    rng = np.random.default_rng(1000 + seed)
    L = int(rng.integers(40, 400))
    d = 128 if seed % 3 == 0 else 64
    dtype = "bf16" if seed % 2 == 0 else "f32"
    terms = _random_terms(rng, L)
    print(f"[gpu] random descriptor seed={seed} L={L} d={d} {dtype} terms={terms}", flush=True)
    M = om.terms_mask(L, terms)
    try:
        a = splat.Acsr(splat.Pattern.from_terms(L, terms))
    except splat.SplatError as e:
        assert e.name == "UNSUPPORTED"   # a row would need more runs than the format holds
        pytest.skip(f"seed {seed}: {e}")
    w = workloads.Workload("random_terms", 1, 2, L, d, dtype, ("terms", ()), 1.0, 2000 + seed)
    Q, K, V = workloads.make_qkv(w)
    ref, Sref, Pref = oa.masked_attention(Q, K, V, M, w.scale, want_csr=True)
    Qd, Kd, Vd = _dev(Q), _dev(K), _dev(V)
    O32 = splat.sparse_mhsa_fwd(a, Qd, Kd, Vd, w.scale, out_dtype=torch.float32)
    O16 = splat.sparse_mhsa_fwd(a, Qd, Kd, Vd, w.scale, out_dtype=torch.bfloat16)
    S, P, Ou = unfused(a, splat, Qd, Kd, Vd, w.scale, torch.float32)
    torch.cuda.synchronize()
    check_O(O32, ref, dtype, f"seed {seed} fused")
    check_O(O16, ref, "bf16", f"seed {seed} fused out=bf16")
    check_O(Ou, ref, dtype, f"seed {seed} unfused")
    rp, ci = om.csr(M)
    q, k = oa.to_f64(Q), oa.to_f64(K)
    S, P = S.cpu().numpy(), P.cpu().numpy()
    for h in range(2):
        assert _s_err_csr(S[0, h], Sref[0, h], q[0, h], k[0, h], rp, ci, w.scale) <= S_REL
        if Pref[0, h].size:
            assert np.abs(P[0, h] - Pref[0, h]).max() <= P_ABS


@pytest.mark.parametrize("seed", range(6))
def test_random_descriptor_patterns_large(gpu_lib, seed):
    """Random patterns over many tiles and row groups (L = 1000 .. 3000), with
    a ragged last group, against the dense oracle."""
    splat = gpu_lib
    rng = np.random.default_rng(5000 + seed)
    L = int(rng.integers(1000, 3000))
    d = 128 if seed % 2 else 64
    dtype = "f32" if seed == 5 else "bf16"
    for _ in range(20):     # redraw until every row fits the format's runs
        terms = _random_terms(rng, L)
        try:
            a = splat.Acsr(splat.Pattern.from_terms(L, terms))
            break
        except splat.SplatError as e:
            assert e.name == "UNSUPPORTED"
    else:
        pytest.fail("no buildable pattern in 20 draws")
    print(f"[gpu] large random descriptor seed={seed} L={L} d={d} {dtype} terms={terms}", flush=True)
    M = om.terms_mask(L, terms)
    w = workloads.Workload("random_terms_large", 1, 2, L, d, dtype, ("terms", ()), 1.0, 6000 + seed)
    Q, K, V = workloads.make_qkv(w)
    ref = oa.masked_attention(Q, K, V, M, w.scale)
    Qd, Kd, Vd = _dev(Q), _dev(K), _dev(V)
    O = splat.sparse_mhsa_fwd(a, Qd, Kd, Vd, w.scale, out_dtype=torch.float32)
    _, _, Ou = unfused(a, splat, Qd, Kd, Vd, w.scale, torch.float32)
    torch.cuda.synchronize()
    check_O(O, ref, dtype, f"seed {seed} fused")
    check_O(Ou, ref, dtype, f"seed {seed} unfused")


# --------------------------------------------------------------------------
# handles built by the paper's analysis pass on explicit masks (two-point
# affine solve per row, regularity check), through both paths
@pytest.mark.parametrize("kind,params,L,d,dtype", [
    ("window", {"w": 37}, 300, 64, "bf16"),
    ("dilated", {"w": 20, "dilation": 3}, 257, 128, "bf16"),
    ("blocked", {"block": 32}, 200, 64, "f32"),
    ("full", {}, 130, 64, "bf16"),
])
def test_from_mask_handles(gpu_lib, kind, params, L, d, dtype):
    splat = gpu_lib
    print(f"[gpu] from_mask {kind} {params} L={L} d={d} {dtype}", flush=True)
    M = om.dense_mask(kind, params, L)
    a = splat.Acsr(mask=M)
    w = workloads.Workload("from_mask", 2, 2, L, d, dtype, workloads.make_pattern(kind, **params),
                           1.0, 31 + L)
    Q, K, V = workloads.make_qkv(w)
    ref, Sref, Pref = oa.masked_attention(Q, K, V, M, w.scale, want_csr=True)
    Qd, Kd, Vd = _dev(Q), _dev(K), _dev(V)
    O = splat.sparse_mhsa_fwd(a, Qd, Kd, Vd, w.scale, out_dtype=torch.float32)
    S, P, Ou = unfused(a, splat, Qd, Kd, Vd, w.scale, torch.float32)
    torch.cuda.synchronize()
    check_O(O, ref, dtype, "fused")
    check_O(Ou, ref, dtype, "unfused")
    rp, ci = om.csr(M)
    q, k = oa.to_f64(Q), oa.to_f64(K)
    S, P = S.cpu().numpy(), P.cpu().numpy()
    for b in range(2):
        for h in range(2):
            assert _s_err_csr(S[b, h], Sref[b, h], q[b, h], k[b, h], rp, ci, w.scale) <= S_REL
            assert np.abs(P[b, h] - Pref[b, h]).max() <= P_ABS


# row softmax on its own, every kernel variant: LPR lanes per row for rows of
# at most 4 LPR values (LPR = 1 .. 32, with rows that fill their lanes
# exactly), a wavefront per row up to 2048 values, two passes beyond
SOFTMAX_ROWS = [
    ("window", {"w": 0}, 77), ("blocked", {"block": 2}, 300), ("window", {"w": 3}, 129),
    ("blocked", {"block": 4}, 257), ("window", {"w": 7}, 1000), ("blocked", {"block": 16}, 333),
    ("window", {"w": 31}, 700), ("window", {"w": 63}, 520), ("window", {"w": 100}, 700),
    ("window", {"w": 300}, 900), ("window", {"w": 700}, 1500), ("window", {"w": 2100}, 4300),
]


@pytest.mark.parametrize("kind,params,L", SOFTMAX_ROWS)
def test_softmax_row_lengths(gpu_lib, kind, params, L):
    splat = gpu_lib
    a = splat.Acsr(splat.Pattern.named(kind, params, L))
    rp, _ = a.export()
    print(f"[gpu] softmax {kind} {params} L={L} max row {a.info()['max_row_nnz']}", flush=True)
    S = workloads.make_scores(2, 3, a.nnz, seed=L + 7)
    P = torch.full_like(S, float("nan")).cuda()
    splat.row_softmax(a, S.cuda(), P)
    torch.cuda.synchronize()
    P = P.cpu().numpy()
    for b in range(2):
        for h in range(3):
            err = np.abs(P[b, h] - oa.softmax_csr(S[b, h], rp)).max()
            assert err <= P_ABS, f"head {(b, h)}: {err:.3e}"


def test_softmax_rows_times_heads_beyond_32bit_grid(gpu_lib):
    """B*H*L = 1040 * 65536 rows of 2-3 values: a grid of 64 lanes per row in
    one dimension would need 4.4e9 work-items."""
    splat = gpu_lib
    B, H, L = 8, 130, 65536
    a = splat.Acsr(splat.Pattern.window(L, 1))
    rp, _ = a.export()
    print(f"[gpu] softmax B*H={B * H} L={L} nnz={a.nnz}", flush=True)
    S = workloads.make_scores(B, H, a.nnz, seed=41)
    Sd = S.cuda()
    P = torch.full_like(Sd, float("nan"))
    splat.row_softmax(a, Sd, P)
    counts = torch.from_numpy(np.diff(rp)).long().cuda()
    row_of = torch.repeat_interleave(torch.arange(L, device="cuda"), counts)
    sums = torch.zeros((B * H, L), dtype=torch.float64, device="cuda")
    sums.index_add_(1, row_of, P.view(B * H, -1).double())
    torch.cuda.synchronize()
    assert torch.isfinite(P).all(), "every value of every row and head is written"
    assert (sums - 1).abs().max().item() <= 1e-5
    for b, h in ((0, 0), (3, 77), (B - 1, H - 1)):
        for i in (0, 1, 4097, L - 2, L - 1):
            seg = slice(int(rp[i]), int(rp[i + 1]))
            ref = oa.softmax_csr(S[b, h, seg], [0, seg.stop - seg.start])
            assert np.abs(P[b, h, seg].cpu().numpy() - ref).max() <= P_ABS


def test_bf16_launch_limit_is_an_error(gpu_lib):
    """A bf16 call whose plan needs more than 2^24 (row group, batch*head)
    workgroups is refused before anything is launched."""
    splat = gpu_lib
    import ctypes
    lib = splat.load()
    a = splat.Acsr(splat.Pattern.window(40000, 1))
    groups = a.info()["n_groups"]
    B, H = 5, 13107                              # B*H = 65535
    assert groups * B * H * 256 > 2 ** 32
    buf = torch.zeros(1024, dtype=torch.float32, device="cuda")
    p = ctypes.c_void_p(buf.data_ptr())
    st = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    assert lib.splat_rsddmm(a.handle, 1, B, H, 64, p, p, ctypes.c_float(0.125), p, st) == 2
    assert b"workgroups" in lib.splat_last_error()
    assert lib.splat_rspmm(a.handle, 1, B, H, 64, p, p, p, 1, st) == 2
    assert lib.splat_sparse_mhsa_fwd(a.handle, 1, B, H, 64, p, p, p, ctypes.c_float(0.125), p, 1,
                                     st) == 2
    torch.cuda.synchronize()


# Score regimes of the bf16 fused kernel's online softmax, one per head: the
# reference rising over many tiles, scores far above and far below the range
# its fast pass applies ([0, 100] in log2 units), and rows whose exponentials
# start in the fp32 subnormal band.  q and k lie along one direction, so the
# scores are set by their lengths; t = scale*log2(e)*q.k.
REGIMES = {
    "rising to ~280": (2.0, lambda c: 12.0 * c),
    "near +400": (5.0, lambda c: 7.0 + 0 * c),
    "near -400": (5.0, lambda c: -7.0 + 0 * c),
    "near -120": (2.0, lambda c: -5.2 + 0 * c),
    "falling from ~100 to -300": (2.0, lambda c: 4.3 - 17.3 * c),
}


@pytest.mark.parametrize("kind,params,L,d", [("window", {"w": 300}, 700, 64),
                                             ("window_global", {"w": 100, "n_global": 9}, 515, 64),
                                             ("window", {"w": 200}, 450, 128)])
def test_fused_score_regimes(gpu_lib, kind, params, L, d):
    splat = gpu_lib
    H = len(REGIMES)
    scale = 1.0 / math.sqrt(d)
    g = torch.Generator().manual_seed(L)
    # |u|^2 * scale = 8 at every d, so each regime keeps its score range
    u = torch.full((d,), math.sqrt(8.0 / (scale * d)), dtype=torch.float64)
    c = torch.arange(L, dtype=torch.float64) / L
    Q = torch.empty(1, H, L, d, dtype=torch.float64)
    K = torch.empty_like(Q)
    for h, (qa, kf) in enumerate(REGIMES.values()):
        Q[0, h] = qa * u + 0.05 * torch.randn(L, d, generator=g, dtype=torch.float64)
        K[0, h] = kf(c)[:, None] * u + 0.3 * torch.randn(L, d, generator=g, dtype=torch.float64)
    V = torch.randn(1, H, L, d, generator=g, dtype=torch.float64)
    Q, K, V = (x.to(torch.bfloat16) for x in (Q, K, V))
    print(f"[gpu] score regimes {kind} {params} L={L} d={d}", flush=True)
    M = om.dense_mask(kind, params, L)
    ref = oa.masked_attention(Q, K, V, M, scale)
    a = splat.Acsr(splat.Pattern.named(kind, params, L))
    Qd, Kd, Vd = _dev(Q), _dev(K), _dev(V)
    O = splat.sparse_mhsa_fwd(a, Qd, Kd, Vd, scale, out_dtype=torch.float32)
    Ob = splat.sparse_mhsa_fwd(a, Qd, Kd, Vd, scale)
    torch.cuda.synchronize()
    for h, name in enumerate(REGIMES):
        check_O(O[:, h:h + 1], ref[:, h:h + 1], "bf16", f"fused, {name}")
        check_O(Ob[:, h:h + 1], ref[:, h:h + 1], "bf16", f"fused bf16 out, {name}")


def test_many_heads(gpu_lib):
    """B*H = 600 (not a power of two): the workgroup -> (row group, head) split."""
    splat = gpu_lib
    w = workloads.Workload("many_heads", 15, 40, 192, 64, "bf16",
                           workloads.make_pattern("window_global", w=20, n_global=3), 1.0, 77)
    print(f"[gpu] many heads B={w.B} H={w.H} L={w.L}", flush=True)
    Q, K, V = workloads.make_qkv(w)
    M = om.dense_mask(w.kind, w.params, w.L)
    ref = oa.masked_attention(Q, K, V, M, w.scale)
    a = splat.Acsr(splat.Pattern.named(w.kind, w.params, w.L))
    Qd, Kd, Vd = _dev(Q), _dev(K), _dev(V)
    O = splat.sparse_mhsa_fwd(a, Qd, Kd, Vd, w.scale, out_dtype=torch.float32)
    _, _, Ou = unfused(a, splat, Qd, Kd, Vd, w.scale, torch.float32)
    torch.cuda.synchronize()
    check_O(O, ref, "bf16", "fused")
    check_O(Ou, ref, "bf16", "unfused")


def test_maximum_length(gpu_lib):
    """L = SPLAT_MAX_L = 65536 with a thin window: index arithmetic at the
    largest size, checked on sampled rows (a dense oracle mask would be 4 GiB)."""
    splat = gpu_lib
    L = 65536
    w = workloads.Workload("max_len", 1, 2, L, 64, "bf16", workloads.make_pattern("window", w=24),
                           1.0, 99)
    print(f"[gpu] maximum length L={L}", flush=True)
    Q, K, V = workloads.make_qkv(w)
    a = splat.Acsr(splat.Pattern.named(w.kind, w.params, w.L))
    Qd, Kd, Vd = _dev(Q), _dev(K), _dev(V)
    O = splat.sparse_mhsa_fwd(a, Qd, Kd, Vd, w.scale, out_dtype=torch.float32)
    _, _, Ou = unfused(a, splat, Qd, Kd, Vd, w.scale, torch.float32)
    torch.cuda.synchronize()
    O, Ou = O.cpu().numpy(), Ou.cpu().numpy()
    rng = np.random.default_rng(5)
    rows = _sample_rows(L, [0, 1, 23, 24, 25, 32767, 32768, L - 26, L - 25, L - 1], rng, 30)
    cols = om.row_columns_fast(w.kind, w.params, L, rows)
    q, k, v = oa.to_f64(Q), oa.to_f64(K), oa.to_f64(V)
    for h in range(2):
        _, _, Or = oa.attention_rows(q[0, h], k[0, h], v[0, h], rows, cols, w.scale)
        for name, X in (("fused", O), ("unfused", Ou)):
            err = float(np.abs(X[0, h, rows] - Or).max())
            assert err <= BF16_ABS, f"{name} head {h}: {err:.3e}"
