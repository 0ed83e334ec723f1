"""Sparse multi-head self-attention over ACSR masks on MI355X (gfx950).

Thin Python binding of ``libsplat.so`` (C ABI in ``include/splat.h``): this
module only marshals arguments -- PyTorch supplies device memory and the
stream, every step of the computation runs in the library's HIP kernels.
There is no fallback: if the library is not built, ``load()`` raises.

    import paper_2407_16847_amd as splat
    pat = splat.Pattern.window_global(4096, w=512, n_global=64)
    acsr = splat.Acsr(pat)                       # host analysis + device upload
    O = splat.sparse_mhsa_fwd(acsr, Q, K, V, scale)   # fused forward
    S = splat.rsddmm(acsr, Q, K, scale)          # unfused: SDDMM
    P = splat.row_softmax(acsr, S)               #          softmax over non-zeros
    O = splat.rspmm(acsr, P, V)                  #          SpMM
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Tuple

import numpy as np
import torch  # loaded first: libsplat then binds to the HIP runtime torch uses

__all__ = [
    "SplatError", "Pattern", "Acsr", "load", "lib_path", "rsddmm", "row_softmax", "rspmm",
    "sparse_mhsa_fwd", "MAX_RUNS", "MAX_TERMS", "PLAN_NO_SPAN", "NO_SPAN_MAX_L", "PLAN_COLUMNS",
    "DENSE_ALPHA", "transpose_colmajor", "rspmm_colmajor", "sparse_mhsa_unfused",
]

MAX_TERMS = 8
MAX_RUNS = 4
PLAN_NO_SPAN = 1          # SPLAT_PLAN_NO_SPAN
PLAN_COLUMNS = 2          # SPLAT_PLAN_COLUMNS
DENSE_ALPHA = 0.10        # SPLAT_DENSE_ALPHA
NO_SPAN_MAX_L = 16384     # SPLAT_NO_SPAN_MAX_L
F32, BF16 = 0, 1
_STATUS = {0: "OK", 1: "INVALID_ARG", 2: "UNSUPPORTED", 3: "NOT_REGULAR", 4: "OOM", 5: "HIP",
           6: "NO_DEVICE"}


class SplatError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"SPLAT_ERR_{_STATUS.get(status, status)}: {message}")
        self.status = status
        self.name = _STATUS.get(status, str(status))


class AffineTerm(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("row_lo", "row_hi", "group", "lo_i", "lo_q", "lo_c", "hi_i", "hi_q", "hi_c", "stride")]


class PatternDesc(ctypes.Structure):
    _fields_ = [("L", ctypes.c_int32), ("n_terms", ctypes.c_int32), ("terms", AffineTerm * MAX_TERMS)]


class AcsrInfo(ctypes.Structure):
    _fields_ = [("L", ctypes.c_int32), ("max_row_nnz", ctypes.c_int32), ("max_runs", ctypes.c_int32),
                ("on_device", ctypes.c_int32), ("device", ctypes.c_int32), ("bm", ctypes.c_int32),
                ("bn", ctypes.c_int32), ("n_groups", ctypes.c_int32), ("n_tiles", ctypes.c_int32),
                ("n_full_tiles", ctypes.c_int32), ("nnz", ctypes.c_int64), ("computed", ctypes.c_int64),
                ("columns", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class TilingStats(ctypes.Structure):
    _fields_ = [("blocks", ctypes.c_int64), ("points", ctypes.c_int64), ("divergent", ctypes.c_int64),
                ("redundant", ctypes.c_int64), ("reuse", ctypes.c_double),
                ("coalesced", ctypes.c_double), ("cost", ctypes.c_double),
                ("stretch", ctypes.c_int32), ("iterations", ctypes.c_int32)]


TILING_METHODS = {"poset": 0, "grid": 1, "naive": 2}

_LIB: Optional[ctypes.CDLL] = None
_LIB_CHECKED: Optional[ctypes.CDLL] = None


def lib_path(checked: bool = False) -> str:
    name = "libsplat_checked.so" if checked else "libsplat.so"
    return os.path.join(os.path.dirname(os.path.abspath(__file__)), name)


def load() -> ctypes.CDLL:
    """Load libsplat.so (built in-tree).  Raises if it is missing."""
    global _LIB
    if _LIB is None:
        _LIB = _open(lib_path())
    return _LIB


def load_checked() -> ctypes.CDLL:
    """Load libsplat_checked.so, the build with device-side index checks (a
    debugging aid: the same C ABI, its kernels checking every index they derive
    from the plan; see splat_debug_bounds).  The module's own calls keep using
    libsplat.so; the checked library is driven through its C ABI directly."""
    global _LIB_CHECKED
    if _LIB_CHECKED is None:
        _LIB_CHECKED = _open(lib_path(checked=True))
    return _LIB_CHECKED


def _open(path: str) -> ctypes.CDLL:
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built; run `python -m paper_2407_16847_amd.build` "
                           "(or __graft_entry__.build()) first")
    lib = ctypes.CDLL(path)
    i32, i64, vp, f32 = ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p, ctypes.c_float
    P = ctypes.POINTER
    sig = {
        "splat_pattern_window": [i32, i32, P(PatternDesc)],
        "splat_pattern_blocked": [i32, i32, P(PatternDesc)],
        "splat_pattern_strided_local": [i32, i32, i32, P(PatternDesc)],
        "splat_pattern_dilated": [i32, i32, i32, P(PatternDesc)],
        "splat_pattern_window_global": [i32, i32, i32, P(PatternDesc)],
        "splat_pattern_full": [i32, P(PatternDesc)],
        "splat_acsr_build": [P(PatternDesc), P(vp)],
        "splat_acsr_build_ex": [P(PatternDesc), ctypes.c_uint32, P(vp)],
        "splat_acsr_from_mask": [i32, vp, P(vp)],
        "splat_acsr_info": [vp, P(AcsrInfo)],
        "splat_acsr_export": [vp, vp, vp],
        "splat_acsr_row_runs": [vp, i32, vp, P(i32)],
        "splat_acsr_export_plan": [vp, vp, vp, vp],
        "splat_acsr_tile_row_mask": [vp, i32, i32, P(ctypes.c_uint64)],
        "splat_rsddmm": [vp, i32, i32, i32, i32, vp, vp, f32, vp, vp],
        "splat_row_softmax": [vp, i32, i32, vp, vp, vp],
        "splat_rspmm": [vp, i32, i32, i32, i32, vp, vp, vp, i32, vp],
        "splat_sparse_mhsa_fwd": [vp, i32, i32, i32, i32, vp, vp, vp, f32, vp, i32, vp],
        "splat_sparse_mhsa_unfused_noalloc": [vp, i32, i32, i32, i32, vp, vp, vp, f32, vp, i32, f32,
                                              P(i32), vp],
        "splat_acsr_export_csc": [vp, vp, vp],
        "splat_acsr_tiling": [vp, i32, i32, i32, i32, P(TilingStats), vp, i64],
        "splat_transpose_colmajor": [vp, i32, i32, vp, vp, vp],
        "splat_rspmm_colmajor": [vp, i32, i32, i32, i32, vp, vp, vp, i32, vp],
        "splat_sparse_mhsa_unfused": [vp, i32, i32, i32, i32, vp, vp, vp, f32, vp, vp, vp, i32, f32,
                                      P(i32), vp],
        "splat_debug_bounds": [P(ctypes.c_uint32), i32],
        "splat_debug_bounds_probe": [i32, i32, i32, P(i32)],
    }
    for name, args in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = ctypes.c_int
    lib.splat_acsr_destroy.argtypes = [vp]
    lib.splat_acsr_destroy.restype = None
    lib.splat_last_error.restype = ctypes.c_char_p
    lib.splat_version.restype = ctypes.c_char_p
    return lib


def _check(status: int) -> None:
    if status != 0:
        msg = load().splat_last_error().decode(errors="replace")
        raise SplatError(status, msg)


# ---------------------------------------------------------------------------
class Pattern:
    """A pattern descriptor (union of affine terms, see include/splat.h)."""

    def __init__(self, desc: PatternDesc):
        self.desc = desc

    @property
    def L(self) -> int:
        return int(self.desc.L)

    @classmethod
    def _make(cls, fn: str, *args) -> "Pattern":
        d = PatternDesc()
        _check(getattr(load(), fn)(*args, ctypes.byref(d)))
        return cls(d)

    @classmethod
    def window(cls, L, w):
        return cls._make("splat_pattern_window", L, w)

    @classmethod
    def blocked(cls, L, block):
        return cls._make("splat_pattern_blocked", L, block)

    @classmethod
    def strided_local(cls, L, local, stride):
        return cls._make("splat_pattern_strided_local", L, local, stride)

    @classmethod
    def dilated(cls, L, w, dilation):
        return cls._make("splat_pattern_dilated", L, w, dilation)

    @classmethod
    def window_global(cls, L, w, n_global):
        return cls._make("splat_pattern_window_global", L, w, n_global)

    @classmethod
    def full(cls, L):
        return cls._make("splat_pattern_full", L)

    @classmethod
    def from_terms(cls, L: int, terms) -> "Pattern":
        """terms: iterable of dicts with the AffineTerm field names (defaults:
        rows [0, L), group 1, stride 1, coefficients 0)."""
        d = PatternDesc()
        d.L = L
        terms = list(terms)
        if len(terms) > MAX_TERMS:
            raise ValueError(f"at most {MAX_TERMS} terms")
        d.n_terms = len(terms)
        for k, t in enumerate(terms):
            base = dict(row_lo=0, row_hi=L, group=1, lo_i=0, lo_q=0, lo_c=0, hi_i=0, hi_q=0, hi_c=0,
                        stride=1)
            base.update(t)
            for f, v in base.items():
                setattr(d.terms[k], f, int(v))
        return cls(d)

    @classmethod
    def named(cls, kind: str, params: dict, L: int) -> "Pattern":
        """A workload pattern by kind name and parameters."""
        p = dict(params)
        if kind == "window":
            return cls.window(L, p["w"])
        if kind == "blocked":
            return cls.blocked(L, p["block"])
        if kind == "strided_local":
            return cls.strided_local(L, p["local"], p["stride"])
        if kind == "dilated":
            return cls.dilated(L, p["w"], p["dilation"])
        if kind == "window_global":
            return cls.window_global(L, p["w"], p["n_global"])
        if kind == "full":
            return cls.full(L)
        raise ValueError(f"unknown pattern kind {kind!r}")


class Acsr:
    """An ACSR handle: per-row affine runs + work plan, on the current device."""

    def __init__(self, pattern: Optional[Pattern] = None, *, mask: Optional[np.ndarray] = None,
                 span: bool = True, columns: bool = False):
        """span=False plans without span specialisation (every group walks all
        of [0, L); an ablation).  columns=True adds the column-wise analysis
        (the column-major layout when every column is one affine run).  Both
        need a pattern, not a mask."""
        lib = load()
        h = ctypes.c_void_p()
        flags = (0 if span else PLAN_NO_SPAN) | (PLAN_COLUMNS if columns else 0)
        if mask is not None:
            if flags:
                raise ValueError("span=False and columns=True need a pattern, not a mask")
            m = np.ascontiguousarray(np.asarray(mask, dtype=np.uint8))
            if m.ndim != 2 or m.shape[0] != m.shape[1]:
                raise ValueError("mask must be a square [L, L] array")
            _check(lib.splat_acsr_from_mask(int(m.shape[0]), m.ctypes.data_as(ctypes.c_void_p),
                                            ctypes.byref(h)))
        else:
            if pattern is None:
                raise ValueError("need a pattern or a mask")
            if flags == 0:
                _check(lib.splat_acsr_build(ctypes.byref(pattern.desc), ctypes.byref(h)))
            else:
                _check(lib.splat_acsr_build_ex(ctypes.byref(pattern.desc), flags, ctypes.byref(h)))
        self._h = h
        self._lib = lib
        self._info = self.info()

    def close(self) -> None:
        if getattr(self, "_h", None) is not None and self._h.value:
            self._lib.splat_acsr_destroy(self._h)
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    @property
    def handle(self) -> ctypes.c_void_p:
        if not self._h.value:
            raise ValueError("ACSR handle is closed")
        return self._h

    def info(self) -> dict:
        inf = AcsrInfo()
        _check(self._lib.splat_acsr_info(self.handle, ctypes.byref(inf)))
        return {f: getattr(inf, f) for f, _ in AcsrInfo._fields_}

    @property
    def L(self) -> int:
        return int(self._info["L"])

    @property
    def nnz(self) -> int:
        return int(self._info["nnz"])

    def export(self) -> Tuple[np.ndarray, np.ndarray]:
        rp = np.zeros(self.L + 1, dtype=np.int32)
        ci = np.zeros(max(self.nnz, 1), dtype=np.int32)
        _check(self._lib.splat_acsr_export(self.handle, rp.ctypes.data_as(ctypes.c_void_p),
                                           ci.ctypes.data_as(ctypes.c_void_p)))
        return rp, ci[: self.nnz]

    def export_csc(self) -> Tuple[np.ndarray, np.ndarray]:
        """(col_ptr [L+1], row_idx [nnz]): the column-major value order."""
        cp = np.zeros(self.L + 1, dtype=np.int32)
        ri = np.zeros(max(self.nnz, 1), dtype=np.int32)
        _check(self._lib.splat_acsr_export_csc(self.handle, cp.ctypes.data_as(ctypes.c_void_p),
                                               ri.ctypes.data_as(ctypes.c_void_p)))
        return cp, ri[: self.nnz]

    def tiling(self, method: str = "poset", m: int = 32, n: int = 32, stretch: int = 0,
               anchors: bool = False):
        """Thread-block arrangement statistics under the cost model of
        section 7 (dict); with anchors=True also the (row, col) anchors
        [blocks, 2] in placement order."""
        st = TilingStats()
        _check(self._lib.splat_acsr_tiling(self.handle, TILING_METHODS[method], m, n, stretch,
                                           ctypes.byref(st), None, 0))
        out = {f: getattr(st, f) for f, _ in TilingStats._fields_}
        if not anchors:
            return out
        buf = np.zeros((max(st.blocks, 1), 2), dtype=np.int32)
        _check(self._lib.splat_acsr_tiling(self.handle, TILING_METHODS[method], m, n, stretch,
                                           ctypes.byref(st), buf.ctypes.data_as(ctypes.c_void_p),
                                           st.blocks))
        return out, buf[: st.blocks]

    def row_runs(self, row: int):
        buf = np.zeros(3 * MAX_RUNS, dtype=np.int32)
        n = ctypes.c_int32()
        _check(self._lib.splat_acsr_row_runs(self.handle, int(row), buf.ctypes.data_as(ctypes.c_void_p),
                                             ctypes.byref(n)))
        return [tuple(int(x) for x in buf[3 * r:3 * r + 3]) for r in range(n.value)]

    def export_plan(self):
        inf = self.info()
        g = np.zeros((inf["n_groups"], 4), dtype=np.int32)
        rows = np.zeros(self.L, dtype=np.int32)
        t = np.zeros((max(inf["n_tiles"], 1), 5), dtype=np.int32)
        _check(self._lib.splat_acsr_export_plan(self.handle, g.ctypes.data_as(ctypes.c_void_p),
                                                rows.ctypes.data_as(ctypes.c_void_p),
                                                t.ctypes.data_as(ctypes.c_void_p)))
        return g, rows, t[: inf["n_tiles"]]

    def tile_row_mask(self, tile: int, row: int) -> int:
        b = ctypes.c_uint64()
        _check(self._lib.splat_acsr_tile_row_mask(self.handle, int(tile), int(row), ctypes.byref(b)))
        return int(b.value)


# ---------------------------------------------------------------------------
_DT = {torch.float32: F32, torch.bfloat16: BF16}


def _dense(x: torch.Tensor, name: str, acsr: Acsr, d: Optional[int] = None):
    if not isinstance(x, torch.Tensor) or not x.is_cuda:
        raise TypeError(f"{name} must be a CUDA (HIP) tensor")
    if x.dtype not in _DT:
        raise TypeError(f"{name} must be float32 or bfloat16, got {x.dtype}")
    if x.dim() != 4 or x.shape[2] != acsr.L:
        raise ValueError(f"{name} must be [B, H, L={acsr.L}, d], got {tuple(x.shape)}")
    if d is not None and x.shape[3] != d:
        raise ValueError(f"{name} has d={x.shape[3]}, expected {d}")
    if not x.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return x


def _on(x: torch.Tensor, name: str, ref: torch.Tensor, shape=None) -> None:
    """x lives on ref's device (and has `shape`, when given)."""
    if x.device != ref.device:
        raise ValueError(f"{name} is on {x.device}, expected {ref.device}")
    if shape is not None and tuple(x.shape) != tuple(shape):
        raise ValueError(f"{name} must be {tuple(shape)}, got {tuple(x.shape)}")


def _stream() -> ctypes.c_void_p:
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _out_dtype(dtype: Optional[torch.dtype], default: torch.dtype) -> torch.dtype:
    dt = default if dtype is None else dtype
    if dt not in _DT:
        raise TypeError("out_dtype must be float32 or bfloat16")
    return dt


def rsddmm(acsr: Acsr, Q: torch.Tensor, K: torch.Tensor, scale: float,
           S: Optional[torch.Tensor] = None) -> torch.Tensor:
    """S[b,h,:] = scale * (Q K^T) sampled at the mask, ACSR (CSR) order, fp32."""
    _dense(Q, "Q", acsr)
    B, H, L, d = Q.shape
    _dense(K, "K", acsr, d)
    if K.dtype != Q.dtype or K.shape[:2] != Q.shape[:2]:
        raise ValueError("K must match Q in dtype, B and H")
    _on(K, "K", Q)
    if S is None:
        S = torch.empty((B, H, acsr.nnz), dtype=torch.float32, device=Q.device)
    else:
        _values(S, "S", acsr, B, H)
        _on(S, "S", Q)
    _check(load().splat_rsddmm(acsr.handle, _DT[Q.dtype], B, H, d, Q.data_ptr(), K.data_ptr(),
                               float(scale), S.data_ptr() if S.numel() else None, _stream()))
    return S


def row_softmax(acsr: Acsr, S: torch.Tensor, P: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Softmax over each row's non-zeros; P may be S (in place)."""
    if not isinstance(S, torch.Tensor) or not S.is_cuda:
        raise TypeError("S must be a CUDA (HIP) tensor")
    if S.dtype != torch.float32 or S.dim() != 3 or S.shape[2] != acsr.nnz or not S.is_contiguous():
        raise ValueError(f"S must be a contiguous float32 [B, H, {acsr.nnz}] tensor")
    B, H, _ = S.shape
    if P is None:
        P = torch.empty_like(S)
    else:
        _values(P, "P", acsr, B, H)
        _on(P, "P", S)
    _check(load().splat_row_softmax(acsr.handle, B, H, S.data_ptr() if S.numel() else None,
                                    P.data_ptr() if P.numel() else None, _stream()))
    return P


def rspmm(acsr: Acsr, P: torch.Tensor, V: torch.Tensor, O: Optional[torch.Tensor] = None,
          out_dtype: Optional[torch.dtype] = None) -> torch.Tensor:
    """O = P V with P in ACSR (CSR) order."""
    _dense(V, "V", acsr)
    B, H, L, d = V.shape
    _values(P, "P", acsr, B, H)
    _on(P, "P", V)
    odt = _out_dtype(out_dtype if O is None else O.dtype, V.dtype)
    if O is None:
        O = torch.empty((B, H, L, d), dtype=odt, device=V.device)
    else:
        _dense(O, "O", acsr, d)
        _on(O, "O", V, (B, H, L, d))
    _check(load().splat_rspmm(acsr.handle, _DT[V.dtype], B, H, d, P.data_ptr() if P.numel() else None,
                              V.data_ptr(), O.data_ptr(), _DT[O.dtype], _stream()))
    return O


def sparse_mhsa_fwd(acsr: Acsr, Q: torch.Tensor, K: torch.Tensor, V: torch.Tensor, scale: float,
                    O: Optional[torch.Tensor] = None,
                    out_dtype: Optional[torch.dtype] = None) -> torch.Tensor:
    """Fused O = softmax_nz(scale * M (x) Q K^T) V."""
    _dense(Q, "Q", acsr)
    B, H, L, d = Q.shape
    for n, x in (("K", K), ("V", V)):
        _dense(x, n, acsr, d)
        if x.dtype != Q.dtype or x.shape[:2] != Q.shape[:2]:
            raise ValueError(f"{n} must match Q in dtype, B and H")
        _on(x, n, Q)
    odt = _out_dtype(out_dtype if O is None else O.dtype, Q.dtype)
    if O is None:
        O = torch.empty((B, H, L, d), dtype=odt, device=Q.device)
    else:
        _dense(O, "O", acsr, d)
        _on(O, "O", Q, (B, H, L, d))
    _check(load().splat_sparse_mhsa_fwd(acsr.handle, _DT[Q.dtype], B, H, d, Q.data_ptr(), K.data_ptr(),
                                        V.data_ptr(), float(scale), O.data_ptr(), _DT[O.dtype],
                                        _stream()))
    return O


def _values(x: torch.Tensor, name: str, acsr: Acsr, B: int, H: int) -> None:
    if not isinstance(x, torch.Tensor) or not x.is_cuda:
        raise TypeError(f"{name} must be a CUDA (HIP) tensor")
    if x.dtype != torch.float32 or tuple(x.shape) != (B, H, acsr.nnz) or not x.is_contiguous():
        raise ValueError(f"{name} must be a contiguous float32 [B, H, {acsr.nnz}] tensor")


def transpose_colmajor(acsr: Acsr, P: torch.Tensor, Pt: Optional[torch.Tensor] = None) -> torch.Tensor:
    """P (CSR value order) -> Pt (column-compressed, column-major order)."""
    if P.dim() != 3:
        raise ValueError("P must be [B, H, nnz]")
    B, H, _ = P.shape
    _values(P, "P", acsr, B, H)
    if Pt is None:
        Pt = torch.empty_like(P)
    _values(Pt, "Pt", acsr, B, H)
    _on(Pt, "Pt", P)
    _check(load().splat_transpose_colmajor(acsr.handle, B, H, P.data_ptr() if P.numel() else None,
                                           Pt.data_ptr() if Pt.numel() else None, _stream()))
    return Pt


def rspmm_colmajor(acsr: Acsr, Pt: torch.Tensor, V: torch.Tensor, O: Optional[torch.Tensor] = None,
                   out_dtype: Optional[torch.dtype] = None) -> torch.Tensor:
    """O = P V with P given in the column-major value order."""
    _dense(V, "V", acsr)
    B, H, L, d = V.shape
    _values(Pt, "Pt", acsr, B, H)
    _on(Pt, "Pt", V)
    odt = _out_dtype(out_dtype if O is None else O.dtype, V.dtype)
    if O is None:
        O = torch.empty((B, H, L, d), dtype=odt, device=V.device)
    else:
        _dense(O, "O", acsr, d)
        _on(O, "O", V, (B, H, L, d))
    _check(load().splat_rspmm_colmajor(acsr.handle, _DT[V.dtype], B, H, d,
                                       Pt.data_ptr() if Pt.numel() else None, V.data_ptr(),
                                       O.data_ptr(), _DT[O.dtype], _stream()))
    return O


def sparse_mhsa_unfused(acsr: Acsr, Q: torch.Tensor, K: torch.Tensor, V: torch.Tensor, scale: float,
                        alpha: float = DENSE_ALPHA, S: Optional[torch.Tensor] = None,
                        Pt: Optional[torch.Tensor] = None, O: Optional[torch.Tensor] = None,
                        out_dtype: Optional[torch.dtype] = None):
    """The unfused chain with the density switch; returns (O, used_colmajor).
    S (and, for a column-major run, Pt) are fp32 [B, H, nnz] workspaces."""
    _dense(Q, "Q", acsr)
    B, H, L, d = Q.shape
    for n, x in (("K", K), ("V", V)):
        _dense(x, n, acsr, d)
        if x.dtype != Q.dtype or x.shape[:2] != Q.shape[:2]:
            raise ValueError(f"{n} must match Q in dtype, B and H")
        _on(x, n, Q)
    if S is None:
        S = torch.empty((B, H, acsr.nnz), dtype=torch.float32, device=Q.device)
    _values(S, "S", acsr, B, H)
    _on(S, "S", Q)
    if Pt is None and acsr.info()["columns"] == 1:
        Pt = torch.empty_like(S)
    if Pt is not None:
        _values(Pt, "Pt", acsr, B, H)
        _on(Pt, "Pt", Q)
    odt = _out_dtype(out_dtype if O is None else O.dtype, Q.dtype)
    if O is None:
        O = torch.empty((B, H, L, d), dtype=odt, device=Q.device)
    else:
        _dense(O, "O", acsr, d)
        _on(O, "O", Q, (B, H, L, d))
    used = ctypes.c_int32(-1)
    _check(load().splat_sparse_mhsa_unfused(
        acsr.handle, _DT[Q.dtype], B, H, d, Q.data_ptr(), K.data_ptr(), V.data_ptr(), float(scale),
        S.data_ptr() if S.numel() else None, Pt.data_ptr() if Pt is not None and Pt.numel() else None,
        O.data_ptr(), _DT[O.dtype], float(alpha), ctypes.byref(used), _stream()))
    return O, bool(used.value)


NOALLOC_SCRATCH_BYTES = 64 << 20   # SPLAT_NOALLOC_SCRATCH_BYTES


def sparse_mhsa_unfused_noalloc(acsr: Acsr, Q: torch.Tensor, K: torch.Tensor, V: torch.Tensor,
                                scale: float, alpha: float = DENSE_ALPHA,
                                O: Optional[torch.Tensor] = None,
                                out_dtype: Optional[torch.dtype] = None):
    """The unfused chain with S (and Pt) in the library's fixed scratch
    instead of caller workspaces; returns (O, used_colmajor).  The call itself
    allocates nothing (an O passed in is used as it is)."""
    _dense(Q, "Q", acsr)
    B, H, L, d = Q.shape
    for n, x in (("K", K), ("V", V)):
        _dense(x, n, acsr, d)
        if x.dtype != Q.dtype or x.shape[:2] != Q.shape[:2]:
            raise ValueError(f"{n} must match Q in dtype, B and H")
        _on(x, n, Q)
    odt = _out_dtype(out_dtype if O is None else O.dtype, Q.dtype)
    if O is None:
        O = torch.empty((B, H, L, d), dtype=odt, device=Q.device)
    else:
        _dense(O, "O", acsr, d)
        _on(O, "O", Q, (B, H, L, d))
    used = ctypes.c_int32(-1)
    _check(load().splat_sparse_mhsa_unfused_noalloc(
        acsr.handle, _DT[Q.dtype], B, H, d, Q.data_ptr(), K.data_ptr(), V.data_ptr(), float(scale),
        O.data_ptr(), _DT[O.dtype], float(alpha), ctypes.byref(used), _stream()))
    return O, bool(used.value)
