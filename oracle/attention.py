"""Masked attention in fp64 (oracle; test infrastructure only).

Equation 1 (section 2, sparse attention) computes softmax(M (x) Q K^T) V, the
sampled product (SDDMM) followed by the row softmax and the sparse-dense
product (SpMM); section 6 applies the softmax to each row of the compressed
matrix.  Readings used here:

* the softmax runs over each row's non-zeros only (a masked-out entry takes
  no part, i.e. it is -inf before the exponential, not 0);
* S carries the attention scale: S = scale * Q K^T (the paper's equation has
  no 1/sqrt(d); the scale is an explicit argument, 1/sqrt(d) in every
  workload);
* a row with no non-zero has P = 0 and O = 0.

Inputs are the exact host tensors the GPU receives (bf16 values upcast
exactly), so the oracle measures the GPU path's own rounding only.
"""
from __future__ import annotations

import math
from typing import Iterable, List, Optional, Sequence

import numpy as np


def to_f64(x) -> np.ndarray:
    """torch tensor (fp32 / bf16, any device) or array -> fp64 numpy, exactly."""
    try:
        import torch
        if isinstance(x, torch.Tensor):
            return x.detach().to("cpu", torch.float64).numpy()
    except ImportError:  # pragma: no cover
        pass
    return np.asarray(x, dtype=np.float64)


def attention_head(q: np.ndarray, k: np.ndarray, v: np.ndarray, mask: np.ndarray,
                   scale: float, row_block: int = 512):
    """One (batch, head): returns dense S (fp64, -inf off the mask), P and O.

    q, k, v are [L, d] fp64, mask is [L, L] bool.  Rows are processed in
    blocks only to bound memory; each row's result does not depend on the
    blocking.
    """
    L = q.shape[0]
    S = np.empty((L, L), dtype=np.float64)
    P = np.empty((L, L), dtype=np.float64)
    O = np.empty((L, v.shape[1]), dtype=np.float64)
    for r0 in range(0, L, row_block):
        r1 = min(L, r0 + row_block)
        m = mask[r0:r1]
        s = scale * (q[r0:r1] @ k.T)                     # SDDMM, sampled below
        s = np.where(m, s, -np.inf)
        has = m.any(axis=1)
        mx = np.where(has, s.max(axis=1, initial=-np.inf), 0.0)
        e = np.where(m, np.exp(s - mx[:, None]), 0.0)  # exp(-inf) never taken
        den = e.sum(axis=1)
        p = np.where(has[:, None], e / np.where(has, den, 1.0)[:, None], 0.0)
        S[r0:r1] = s
        P[r0:r1] = p
        O[r0:r1] = p @ v                                 # SpMM
    return S, P, O


def masked_attention(Q, K, V, mask: np.ndarray, scale: float, want_csr: bool = False):
    """All heads of [B, H, L, d] inputs.

    Returns O [B, H, L, d] fp64, and with ``want_csr`` also S and P gathered at
    the mask's non-zeros in CSR order (row by row, ascending column), shaped
    [B, H, nnz] -- the row-compressed row-major ACSR value order.
    """
    q, k, v = to_f64(Q), to_f64(K), to_f64(V)
    B, H, L, d = q.shape
    mask = np.asarray(mask, dtype=bool)
    nnz = int(mask.sum())
    O = np.empty((B, H, L, v.shape[3]), dtype=np.float64)
    Sc = np.empty((B, H, nnz), dtype=np.float64) if want_csr else None
    Pc = np.empty((B, H, nnz), dtype=np.float64) if want_csr else None
    for b in range(B):
        for h in range(H):
            S, P, O[b, h] = attention_head(q[b, h], k[b, h], v[b, h], mask, scale)
            if want_csr:
                Sc[b, h] = S[mask]
                Pc[b, h] = P[mask]
    if want_csr:
        return O, Sc, Pc
    return O


def attention_rows(q: np.ndarray, k: np.ndarray, v: np.ndarray,
                   rows: Sequence[int], cols: Sequence[np.ndarray], scale: float):
    """Selected rows of one head, each from its own column list.

    q, k, v: [L, d] fp64; cols[t] is the ascending column list of rows[t].
    Returns lists of per-row S (at cols), P (at cols) and O ([d]).
    """
    S_out: List[np.ndarray] = []
    P_out: List[np.ndarray] = []
    O_out = np.zeros((len(rows), v.shape[1]), dtype=np.float64)
    for t, (i, c) in enumerate(zip(rows, cols)):
        c = np.asarray(c, dtype=np.int64)
        if c.size == 0:
            S_out.append(np.zeros(0))
            P_out.append(np.zeros(0))
            continue
        s = scale * (k[c] @ q[i])
        e = np.exp(s - s.max())
        p = e / e.sum()
        S_out.append(s)
        P_out.append(p)
        O_out[t] = p @ v[c]
    return S_out, P_out, O_out


def softmax_csr(values, row_ptr) -> np.ndarray:
    """Softmax of each row of a CSR-ordered value array over the row's entries
    (section 6: the softmax applied to every row of the compressed matrix).

    values: [nnz] (any float type), row_ptr: [n_rows + 1].  Returns fp64 [nnz];
    an empty row has no entries and contributes nothing.
    """
    x = to_f64(values)
    out = np.empty_like(x)
    for i in range(len(row_ptr) - 1):
        lo, hi = int(row_ptr[i]), int(row_ptr[i + 1])
        if hi > lo:
            e = np.exp(x[lo:hi] - x[lo:hi].max())
            out[lo:hi] = e / e.sum()
    return out


def brute_force(q, k, v, pred, scale: float):
    """Pure-Python loops with math.exp and math.fsum (tiny inputs only).

    q, k, v: nested lists / arrays [L][d]; pred(i, j) -> bool.  Returns O as a
    list of lists.  Each sum is correctly rounded (fsum), so this is accurate
    to a few ulps and independent of any BLAS.
    """
    L, d = len(q), len(q[0])
    dv = len(v[0])
    out = []
    for i in range(L):
        js = [j for j in range(L) if pred(i, j)]
        if not js:
            out.append([0.0] * dv)
            continue
        s = {j: scale * math.fsum(float(q[i][c]) * float(k[j][c]) for c in range(d)) for j in js}
        mx = max(s.values())
        e = {j: math.exp(s[j] - mx) for j in js}
        den = math.fsum(e.values())
        out.append([math.fsum(e[j] / den * float(v[j][c]) for j in js) for c in range(dv)])
    return out
