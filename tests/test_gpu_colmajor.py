"""GPU: the column-compressed, column-major value layout (section 5.2) and the
unfused chain's density switch (section 9, data-layout reordering).

* splat_transpose_colmajor is a permutation: its output equals P gathered in
  the oracle's column-major order, bit for bit;
* splat_rspmm_colmajor feeds the same values to the same products in the
  same order as splat_rspmm, so the two outputs are equal bit for bit, and
  both are within the tolerance of the oracle (bf16 inputs: 2e-2 absolute;
  fp32 inputs: 1e-5 per-row normwise);
* splat_sparse_mhsa_unfused takes the column-major branch exactly when the
  density reaches alpha and every column is one affine run.
"""
import ctypes

import numpy as np
import pytest
import torch

import workloads
from oracle import attention as oa
from oracle import masks as om

pytestmark = pytest.mark.gpu

BF16_ABS = 2e-2
F32_REL = 1e-5


def _check(O, ref, dtype, what):
    O = O.float().cpu().numpy().astype(np.float64)
    assert np.isfinite(O).all(), what
    if dtype == "bf16":
        err = float(np.abs(O - ref).max())
        assert err <= BF16_ABS, f"{what}: {err:.3e}"
    else:
        num = np.abs(O - ref).max(axis=-1)
        den = np.abs(ref).max(axis=-1)
        err = float((num[den > 0] / den[den > 0]).max())
        assert err <= F32_REL, f"{what}: {err:.3e}"


def _inputs(kind, params, L, d, dtype, seed):
    w = workloads.Workload("colmajor", 2, 3, L, d, dtype, workloads.make_pattern(kind, **params),
                           1.0, seed)
    Q, K, V = workloads.make_qkv(w)
    return w, Q, K, V


COLS = [
    ("window", {"w": 37}, 300, 64, "bf16"),
    ("blocked", {"block": 32}, 257, 128, "bf16"),
    ("strided_local", {"local": 20, "stride": 16}, 333, 64, "f32"),
    ("dilated", {"w": 30, "dilation": 3}, 400, 64, "bf16"),
    ("full", {}, 200, 64, "f32"),
    ("window", {"w": 1000}, 1500, 128, "bf16"),
]


@pytest.mark.parametrize("kind,params,L,d,dtype", COLS)
def test_transpose_and_colmajor_rspmm(gpu_lib, kind, params, L, d, dtype):
    splat = gpu_lib
    print(f"[gpu] colmajor {kind} {params} L={L} d={d} {dtype}", flush=True)
    a = splat.Acsr(splat.Pattern.named(kind, params, L), columns=True)
    assert a.info()["columns"] == 1
    w, Q, K, V = _inputs(kind, params, L, d, dtype, 500 + L)
    M = om.dense_mask(kind, params, L)
    ref = oa.masked_attention(Q, K, V, M, w.scale)
    Qd, Kd, Vd = Q.cuda(), K.cuda(), V.cuda()
    P = splat.row_softmax(a, splat.rsddmm(a, Qd, Kd, w.scale))
    Pt = torch.full_like(P, float("nan"))
    splat.transpose_colmajor(a, P, Pt)
    O_col = splat.rspmm_colmajor(a, Pt, Vd, out_dtype=torch.float32)
    O_row = splat.rspmm(a, P, Vd, out_dtype=torch.float32)
    O_col16 = splat.rspmm_colmajor(a, Pt, Vd, out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    src = torch.from_numpy(om.colmajor_source(M))
    assert torch.equal(Pt.cpu(), P.cpu()[:, :, src]), "transpose is the column-major permutation"
    assert torch.equal(O_col, O_row), "same values, same products, same order"
    _check(O_col, ref, dtype, "column-major R-SpMM")
    _check(O_col16, ref, "bf16", "column-major R-SpMM, bf16 out")


def test_transpose_with_no_span_plan(gpu_lib):
    """The transpose walks the tile plan; a no-span plan (tiles with empty
    wavefronts and zero masks) gives the same permutation."""
    splat = gpu_lib
    L = 700
    pat = splat.Pattern.window(L, 20)
    a = splat.Acsr(pat, columns=True, span=False)
    M = om.dense_mask("window", {"w": 20}, L)
    S = workloads.make_scores(2, 3, a.nnz, seed=9).cuda()
    Pt = splat.transpose_colmajor(a, S)
    torch.cuda.synchronize()
    assert torch.equal(Pt.cpu(), S.cpu()[:, :, torch.from_numpy(om.colmajor_source(M))])


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_unfused_density_switch(gpu_lib, dtype):
    splat = gpu_lib
    L, d = 600, 64
    w, Q, K, V = _inputs("window", {"w": 150}, L, d, dtype, 77)
    M = om.dense_mask("window", {"w": 150}, L)
    ref = oa.masked_attention(Q, K, V, M, w.scale)
    Qd, Kd, Vd = Q.cuda(), K.cuda(), V.cuda()
    pat = splat.Pattern.window(L, 150)
    a = splat.Acsr(pat, columns=True)
    density = a.nnz / L ** 2
    assert 0.10 <= density <= 0.6
    outs = {}
    # alpha travels as a float: stay clear of the density by more than its rounding
    for alpha, want in ((splat.DENSE_ALPHA, True), (density - 1e-4, True), (density + 1e-4, False),
                        (2.0, False)):
        O, used = splat.sparse_mhsa_unfused(a, Qd, Kd, Vd, w.scale, alpha=alpha,
                                            out_dtype=torch.float32)
        assert used == want, (alpha, used)
        outs[alpha] = O
    plain = splat.Acsr(pat)                         # no column analysis: always row-major
    O_plain, used = splat.sparse_mhsa_unfused(plain, Qd, Kd, Vd, w.scale, alpha=0.0,
                                              out_dtype=torch.float32)
    assert not used
    torch.cuda.synchronize()
    for O in outs.values():
        _check(O, ref, dtype, "unfused")
        assert torch.equal(O, O_plain)
    # a mask whose columns are not single runs stays row-major at any alpha
    wg = splat.Acsr(splat.Pattern.window_global(L, 10, 5), columns=True)
    assert wg.info()["columns"] == 0
    Mg = om.dense_mask("window_global", {"w": 10, "n_global": 5}, L)
    Og, used = splat.sparse_mhsa_unfused(wg, Qd, Kd, Vd, w.scale, alpha=0.0, out_dtype=torch.float32)
    torch.cuda.synchronize()
    assert not used
    _check(Og, oa.masked_attention(Q, K, V, Mg, w.scale), dtype, "unfused, window+global")


def test_colmajor_argument_errors(gpu_lib):
    splat = gpu_lib
    lib = splat.load()
    st = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    L = 128
    plain = splat.Acsr(splat.Pattern.window(L, 4))
    cols = splat.Acsr(splat.Pattern.window(L, 4), columns=True)
    irregular = splat.Acsr(splat.Pattern.window_global(L, 4, 2), columns=True)
    P = torch.zeros((1, 1, cols.nnz), dtype=torch.float32, device="cuda")
    Pt = torch.zeros_like(P)
    pp, pt = ctypes.c_void_p(P.data_ptr()), ctypes.c_void_p(Pt.data_ptr())
    assert lib.splat_transpose_colmajor(plain.handle, 1, 1, pp, pt, st) == 1
    assert b"SPLAT_PLAN_COLUMNS" in lib.splat_last_error()
    Pi = torch.zeros((1, 1, irregular.nnz), dtype=torch.float32, device="cuda")
    Pti = torch.zeros_like(Pi)
    assert lib.splat_transpose_colmajor(irregular.handle, 1, 1, ctypes.c_void_p(Pi.data_ptr()),
                                        ctypes.c_void_p(Pti.data_ptr()), st) == 3
    assert lib.splat_transpose_colmajor(cols.handle, 1, 1, pp, pp, st) == 1     # overlapping
    V = torch.zeros((1, 1, L, 64), dtype=torch.bfloat16, device="cuda")
    O = torch.zeros_like(V)
    assert lib.splat_rspmm_colmajor(plain.handle, 1, 1, 1, 64, pt, ctypes.c_void_p(V.data_ptr()),
                                    ctypes.c_void_p(O.data_ptr()), 1, st) == 1
    # the column-major branch of the chain needs Pt; nothing is enqueued without it
    used = ctypes.c_int32(-7)
    q = ctypes.c_void_p(V.data_ptr())
    rc = lib.splat_sparse_mhsa_unfused(cols.handle, 1, 1, 1, 64, q, q, q, ctypes.c_float(0.125), pp,
                                       None, ctypes.c_void_p(O.data_ptr()), 1, ctypes.c_float(0.0),
                                       ctypes.byref(used), st)
    assert rc == 1 and used.value == -7
    torch.cuda.synchronize()
