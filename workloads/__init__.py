"""Seeded synthetic workloads shared by the oracle, the tests and the benchmark.

This module holds only workload *descriptions* (shapes, dtypes, value
distributions, seeds and the name + parameters of each attention mask) and
the generator of the Q/K/V host tensors.  It holds none of the method's
arithmetic: neither the mask predicate nor any attention math lives here.
The oracle (``oracle/``) and the HIP path (``paper_2407_16847_amd``) each turn
a pattern description into a mask with their own, independent code.

Pattern kinds (row i = query, column j = key, both in [0, L)):

``window``         {"w": w}                      |i - j| <= w
``blocked``        {"block": b}                  j in the block of i or in the block before it
``strided_local``  {"local": n, "stride": s}     causal: j in [i-n+1, i], or j = s-1 (mod s) with j <= i
``dilated``        {"w": w, "dilation": g}       j = i + g*k for integer k with |k| <= w
``window_global``  {"w": w, "n_global": G}       |i - j| <= w, or i < G, or j < G
``full``           {}                            every (i, j)

The five benchmark workloads follow the sparse-MHSA patterns the paper
evaluates (windowed, blocked and strided masks, Evaluation, experimental
setup) at moderate densities; they are synthetic by construction, as the
paper's own masks are.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, Tuple

import torch

__all__ = ["Workload", "CONFIGS", "get", "make_qkv", "make_scores", "pattern_kinds"]


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    B: int
    H: int
    L: int
    d: int
    dtype: str            # "f32" or "bf16": the dtype Q/K/V are handed over in
    pattern: Tuple[str, Tuple[Tuple[str, int], ...]]   # (kind, sorted params)
    std: float = 1.0      # Q/K/V entries are N(0, std**2) before the cast
    seed: int = 0
    fused: bool = False   # the workload the fused forward is measured on

    @property
    def kind(self) -> str:
        return self.pattern[0]

    @property
    def params(self) -> Dict[str, int]:
        return dict(self.pattern[1])

    @property
    def scale(self) -> float:
        return 1.0 / math.sqrt(self.d)

    def with_(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


def _pat(kind: str, **params: int):
    return (kind, tuple(sorted(params.items())))


pattern_kinds = ("window", "blocked", "strided_local", "dilated", "window_global", "full")

CONFIGS: Dict[int, Workload] = {
    1: Workload("window16_L256_d64_f32", 1, 1, 256, 64, "f32", _pat("window", w=16), 1.0, 1),
    2: Workload("blocked64_L1024_d64_bf16", 2, 8, 1024, 64, "bf16", _pat("blocked", block=64), 1.0, 2),
    3: Workload("strided128_local128_L2048_d64_bf16", 2, 12, 2048, 64, "bf16",
                _pat("strided_local", local=128, stride=128), 1.0, 3),
    # N(0, 0.5) is read as variance 0.5 (standard deviation sqrt(0.5))
    4: Workload("dilated2_w256_L4096_d128_bf16", 1, 16, 4096, 128, "bf16",
                _pat("dilated", w=256, dilation=2), math.sqrt(0.5), 4),
    5: Workload("window512_global64_L4096_d64_bf16", 4, 16, 4096, 64, "bf16",
                _pat("window_global", w=512, n_global=64), 1.0, 5, fused=True),
}


def get(cfg: int) -> Workload:
    return CONFIGS[cfg]


def make_pattern(kind: str, **params: int):
    """A pattern description usable in ``Workload.with_(pattern=...)``."""
    if kind not in pattern_kinds:
        raise ValueError(f"unknown pattern kind {kind!r}")
    return _pat(kind, **params)


def make_qkv(w: Workload, device: str = "cpu"):
    """Q, K, V as contiguous [B, H, L, d] tensors in the workload's dtype.

    Drawn in the order Q, K, V from ``torch.Generator('cpu').manual_seed(seed)``
    as fp32 N(0, 1), multiplied by ``std`` and, for bf16 workloads, rounded to
    bfloat16 (round to nearest even).  The oracle consumes exactly these
    (rounded) values, upcast to fp64.
    """
    g = torch.Generator("cpu").manual_seed(int(w.seed))
    shape = (w.B, w.H, w.L, w.d)
    out = []
    for _ in range(3):
        x = torch.randn(shape, generator=g, dtype=torch.float32)
        if w.std != 1.0:
            x = x * w.std
        if w.dtype == "bf16":
            x = x.to(torch.bfloat16)
        elif w.dtype != "f32":
            raise ValueError(f"unknown dtype {w.dtype!r}")
        out.append(x.contiguous().to(device))
    return tuple(out)


def make_scores(B: int, H: int, nnz: int, seed: int, std: float = 3.0):
    """Scores [B, H, nnz] fp32 for exercising the row softmax on its own:
    ``torch.Generator('cpu').manual_seed(seed)``, N(0, 1) times ``std``."""
    g = torch.Generator("cpu").manual_seed(int(seed))
    return (torch.randn((B, H, nnz), generator=g, dtype=torch.float32) * std).contiguous()
