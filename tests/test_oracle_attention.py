"""Pins for the oracle's masked attention (CPU only).

Each check is written as a function of an attention implementation so the
same checks can be run against deliberately broken variants of the oracle
(``test_pins_catch_planted_mistakes``): a dropped term, a wrong softmax domain,
a transposed operand or a wrong index must fail at least one pin.
"""
import math

import numpy as np
import pytest
import torch

import workloads
from oracle import attention as oa
from oracle import masks as om

RNG = np.random.default_rng(1234)


def oracle_head(q, k, v, M, scale):
    return oa.attention_head(q, k, v, M, scale)[2]


# --------------------------------------------------------------------------
# pins, each a function of an implementation attn(q, k, v, M, scale) -> O
# --------------------------------------------------------------------------
def pin_brute_force(attn):
    """Pure-Python fsum loops on tiny inputs, every pattern kind."""
    worst = 0.0
    for kind, params in [("window", {"w": 1}), ("blocked", {"block": 2}),
                         ("strided_local", {"local": 2, "stride": 3}),
                         ("dilated", {"w": 1, "dilation": 2}),
                         ("window_global", {"w": 1, "n_global": 2}), ("full", {})]:
        for L, d in [(1, 1), (5, 3), (8, 4)]:
            q, k, v = (RNG.standard_normal((L, d)) for _ in range(3))
            v = v + RNG.standard_normal((L, 1))          # V columns differ in mean
            scale = 1.0 / math.sqrt(d) if d > 1 else 0.7
            M = om.dense_mask(kind, params, L)
            ref = np.array(oa.brute_force(q.tolist(), k.tolist(), v.tolist(),
                                          om.predicate(kind, params), scale))
            worst = max(worst, float(np.abs(attn(q, k, v, M, scale) - ref).max()))
    return worst <= 1e-13


def pin_rows_sum_to_one(attn):
    """O of V = all-ones is all-ones on every non-empty row (P rows sum to 1)."""
    L, d = 40, 8
    q, k = RNG.standard_normal((L, d)), RNG.standard_normal((L, d))
    M = om.dense_mask("strided_local", {"local": 5, "stride": 6}, L)
    O = attn(q, k, np.ones((L, 3)), M, 0.5)
    return np.abs(O - 1.0).max() <= 1e-12


def pin_zero_query_gives_row_mean(attn):
    """Q = 0: every score is 0, P_ij = 1/nnz_i, O_i = mean of V over row i's columns."""
    L, d = 37, 6
    k, v = RNG.standard_normal((L, d)), RNG.standard_normal((L, 5))
    M = om.dense_mask("window_global", {"w": 3, "n_global": 2}, L)
    O = attn(np.zeros((L, d)), k, v, M, 0.125)
    ref = np.stack([v[M[i]].mean(axis=0) for i in range(L)])
    return np.abs(O - ref).max() <= 1e-13


def pin_full_mask_is_dense_attention(attn):
    """Full mask reduces to dense attention: torch SDPA in fp64 on the CPU."""
    L, d = 24, 8
    q, k, v = (RNG.standard_normal((L, d)) for _ in range(3))
    scale = 1.0 / math.sqrt(d)
    O = attn(q, k, v, np.ones((L, L), dtype=bool), scale)
    t = lambda x: torch.from_numpy(x)[None, None]
    ref = torch.nn.functional.scaled_dot_product_attention(t(q), t(k), t(v), scale=scale)[0, 0].numpy()
    return np.abs(O - ref).max() <= 1e-12


def pin_diagonal_mask_returns_v(attn):
    """A window of width 1 (only j = i) gives P = 1 and O = V exactly."""
    L, d = 19, 4
    q, k, v = (RNG.standard_normal((L, d)) for _ in range(3))
    O = attn(q, k, v, om.dense_mask("window", {"w": 0}, L), 1.0 / math.sqrt(d))
    return np.array_equal(O, v)


def pin_linear_in_v(attn):
    """O(alpha V + beta) = alpha O(V) + beta, because P rows sum to 1."""
    L, d = 30, 4
    q, k, v = (RNG.standard_normal((L, d)) for _ in range(3))
    M = om.dense_mask("dilated", {"w": 3, "dilation": 2}, L)
    a, b = 1.7, -0.3
    lhs = attn(q, k, a * v + b, M, 0.5)
    rhs = a * attn(q, k, v, M, 0.5) + b
    return np.abs(lhs - rhs).max() <= 1e-12


def pin_one_hot_scores(attn):
    """Closed form with two keys: P = softmax([s0, s1]) with s = scale * q.k."""
    q = np.array([[1.0, 0.0], [0.0, 0.0]])
    k = np.array([[2.0, 0.0], [0.0, 5.0]])
    v = np.array([[1.0, 0.0], [0.0, 1.0]])
    M = np.ones((2, 2), dtype=bool)
    O = attn(q, k, v, M, 0.5)
    p0 = math.exp(1.0) / (math.exp(1.0) + 1.0)   # row 0: s = [0.5*2, 0]
    return np.abs(O - np.array([[p0, 1 - p0], [0.5, 0.5]])).max() <= 1e-15


PINS = [pin_brute_force, pin_rows_sum_to_one, pin_zero_query_gives_row_mean,
        pin_full_mask_is_dense_attention, pin_diagonal_mask_returns_v, pin_linear_in_v,
        pin_one_hot_scores]


@pytest.mark.parametrize("pin", PINS, ids=lambda f: f.__name__)
def test_oracle_meets_pin(pin):
    assert pin(oracle_head)


# --------------------------------------------------------------------------
# planted mistakes: each broken variant must fail at least one pin
# --------------------------------------------------------------------------
def _softmax_rows(s):
    e = np.exp(s - s.max(axis=1, keepdims=True))
    return e / e.sum(axis=1, keepdims=True)


def broken_no_scale(q, k, v, M, scale):
    return oa.attention_head(q, k, v, M, 1.0)[2]


def broken_softmax_over_all_entries(q, k, v, M, scale):
    # the literal M (x) QK^T reading: masked entries enter the softmax as 0
    S = np.where(M, scale * q @ k.T, 0.0)
    return (_softmax_rows(S) * M) @ v


def broken_transposed_scores(q, k, v, M, scale):
    S = np.where(M, scale * (k @ q.T), -np.inf)
    return _softmax_rows(S) @ v


def broken_mask_transposed(q, k, v, M, scale):
    return oa.attention_head(q, k, v, np.ascontiguousarray(M.T), scale)[2]


def broken_v_by_row(q, k, v, M, scale):
    P = oa.attention_head(q, k, v, M, scale)[1]
    return P.sum(axis=1, keepdims=True) * v          # row's own V instead of P @ V


def broken_missing_normalisation(q, k, v, M, scale):
    S = np.where(M, scale * q @ k.T, -np.inf)
    E = np.exp(S - S.max(axis=1, keepdims=True))
    return E @ v


def broken_exp_without_max_shift_in_denominator(q, k, v, M, scale):
    S = np.where(M, scale * q @ k.T, -np.inf)
    E = np.exp(S - S.max(axis=1, keepdims=True))
    return (E / np.exp(S).sum(axis=1, keepdims=True)) @ v


BROKEN = [broken_no_scale, broken_softmax_over_all_entries, broken_transposed_scores,
          broken_mask_transposed, broken_v_by_row, broken_missing_normalisation,
          broken_exp_without_max_shift_in_denominator]


@pytest.mark.parametrize("broken", BROKEN, ids=lambda f: f.__name__)
def test_pins_catch_planted_mistakes(broken):
    import warnings
    with warnings.catch_warnings():
        warnings.simplefilter("ignore")
        failed = [p.__name__ for p in PINS if not p(broken)]
    assert failed, f"{broken.__name__} passed every pin"


# --------------------------------------------------------------------------
# the oracle's multi-head, CSR and per-row entry points agree with the head one
# --------------------------------------------------------------------------
def test_csr_export_and_rows_agree_with_dense():
    w = workloads.get(3).with_(B=1, H=2, L=300)
    Q, K, V = workloads.make_qkv(w)
    M = om.dense_mask(w.kind, w.params, w.L)
    O, Sc, Pc = oa.masked_attention(Q, K, V, M, w.scale, want_csr=True)
    row_ptr, col = om.csr(M)
    q, k, v = oa.to_f64(Q), oa.to_f64(K), oa.to_f64(V)
    for h in range(2):
        rows = [0, 1, 127, 128, 255, 256, 299]
        cols = [col[row_ptr[i]:row_ptr[i + 1]] for i in rows]
        S_r, P_r, O_r = oa.attention_rows(q[0, h], k[0, h], v[0, h], rows, cols, w.scale)
        for t, i in enumerate(rows):
            seg = slice(row_ptr[i], row_ptr[i + 1])
            np.testing.assert_allclose(Sc[0, h, seg], S_r[t], rtol=0, atol=1e-13)
            np.testing.assert_allclose(Pc[0, h, seg], P_r[t], rtol=0, atol=1e-15)
            np.testing.assert_allclose(O[0, h, i], O_r[t], rtol=0, atol=1e-13)
            # S in CSR order is scale * q_i . k_j at the listed columns
            np.testing.assert_allclose(Sc[0, h, seg], w.scale * (k[0, h][cols[t]] @ q[0, h, i]),
                                       rtol=0, atol=1e-13)
        assert np.abs(Pc[0, h].sum() - w.L) <= 1e-10


def test_empty_row_gives_zero():
    L = 6
    M = om.dense_mask("window", {"w": 1}, L)
    M[2] = False
    q, k, v = (RNG.standard_normal((L, 3)) for _ in range(3))
    S, P, O = oa.attention_head(q, k, v, M, 0.5)
    assert (O[2] == 0).all() and (P[2] == 0).all()
    assert np.isfinite(O).all()


def test_softmax_csr_pins():
    """softmax_csr against the dense masked path (a -inf mask, not per-row
    slices), scipy's softmax on each row, and closed forms."""
    from scipy.special import softmax as sp_softmax
    w = workloads.get(3).with_(B=1, H=1, L=260)
    Q, K, V = workloads.make_qkv(w)
    M = om.dense_mask(w.kind, w.params, w.L)
    _, Sc, Pc = oa.masked_attention(Q, K, V, M, w.scale, want_csr=True)
    row_ptr, _ = om.csr(M)
    P = oa.softmax_csr(Sc[0, 0], row_ptr)
    np.testing.assert_allclose(P, Pc[0, 0], rtol=0, atol=1e-15)
    for i in (0, 1, 129, 259):
        seg = slice(row_ptr[i], row_ptr[i + 1])
        np.testing.assert_allclose(P[seg], sp_softmax(Sc[0, 0, seg]), rtol=1e-14, atol=0)
    # one entry per row -> exactly 1; equal entries -> 1/n; shift invariance; empty rows
    x = RNG.standard_normal(7)
    assert (oa.softmax_csr(x, np.arange(8)) == 1.0).all()
    assert np.allclose(oa.softmax_csr(np.full(5, 3.25), [0, 5]), 0.2, rtol=0, atol=1e-16)
    v = RNG.standard_normal(9)
    rp = [0, 4, 4, 9]
    np.testing.assert_allclose(oa.softmax_csr(v + 100.0, rp), oa.softmax_csr(v, rp), atol=1e-15)
    out = oa.softmax_csr(v, rp)
    assert abs(out[:4].sum() - 1) < 1e-15 and abs(out[4:].sum() - 1) < 1e-15
