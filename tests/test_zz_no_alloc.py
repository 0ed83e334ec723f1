"""The allocation-free unfused call (splat_sparse_mhsa_unfused_noalloc),
through the C ABI, against splat_sparse_mhsa_unfused with caller workspaces:
the same kernels on the same inputs give the same bits.  Two calls in a row
share the library's scratch, the second on a smaller input (and on the
column-major branch); a request beyond the scratch is refused before any
launch."""
import ctypes

import numpy as np
import pytest
import torch

import workloads
from oracle import attention as oa
from oracle import masks as om

pytestmark = pytest.mark.gpu


def _call_noalloc(lib, a, Q, K, V, scale, O, alpha):
    used = ctypes.c_int32(-1)
    rc = lib.splat_sparse_mhsa_unfused_noalloc(
        a.handle, 1 if Q.dtype == torch.bfloat16 else 0, Q.shape[0], Q.shape[1], Q.shape[3],
        Q.data_ptr(), K.data_ptr(), V.data_ptr(), float(scale), O.data_ptr(),
        1 if O.dtype == torch.bfloat16 else 0, float(alpha), ctypes.byref(used),
        ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    return rc, used.value


def test_noalloc_matches_workspace_call(gpu_lib):
    splat = gpu_lib
    lib = splat.load()
    cases = [
        # B*H*nnz*4 = 25.7 MB of S: strided + local causal mask, row-major branch
        (workloads.get(3), splat.DENSE_ALPHA, torch.float32),
        # a smaller input on the column-major branch (alpha 0): S and Pt
        (workloads.Workload("noalloc_small", 1, 3, 1000, 64, "bf16",
                            workloads.make_pattern("window", w=60), 1.0, 1064), 0.0, torch.bfloat16),
    ]
    for w, alpha, odt in cases:
        print(f"[gpu] noalloc {w.name} B={w.B} H={w.H} L={w.L} alpha={alpha}", flush=True)
        Q, K, V = workloads.make_qkv(w)
        Qd, Kd, Vd = Q.cuda(), K.cuda(), V.cuda()
        a = splat.Acsr(splat.Pattern.named(w.kind, w.params, w.L), columns=True)
        O_ref, used_ref = splat.sparse_mhsa_unfused(a, Qd, Kd, Vd, w.scale, alpha=alpha,
                                                    out_dtype=odt)
        O = torch.full_like(O_ref, float("nan"))
        rc, used = _call_noalloc(lib, a, Qd, Kd, Vd, w.scale, O, alpha)
        torch.cuda.synchronize()
        assert rc == 0, lib.splat_last_error()
        assert used == int(used_ref)
        assert used == (1 if alpha == 0.0 else 0)
        assert torch.equal(O, O_ref), "the allocation-free call differs from the workspace call"
        # and both within the bf16 tolerance of the oracle on every head
        M = om.dense_mask(w.kind, w.params, w.L)
        ref = oa.masked_attention(Q, K, V, M, w.scale)
        err = float(np.abs(O.float().cpu().numpy() - ref).max())
        assert err <= 2e-2, err
        a.close()


def test_noalloc_refuses_requests_beyond_its_scratch(gpu_lib):
    splat = gpu_lib
    lib = splat.load()
    w = workloads.get(5)     # B*H*nnz*4 = 1.12 GB of S
    a = splat.Acsr(splat.Pattern.named(w.kind, w.params, w.L))
    x = torch.zeros((w.B, w.H, w.L, w.d), dtype=torch.bfloat16, device="cuda")
    O = torch.full_like(x, 7.0)
    rc, used = _call_noalloc(lib, a, x, x, x, w.scale, O, splat.DENSE_ALPHA)
    torch.cuda.synchronize()
    assert rc == 2 and b"scratch" in lib.splat_last_error()
    assert used == -1 and bool((O == 7.0).all()), "a refused call wrote its output"
