#!/usr/bin/env python3
"""Density sweep on one MI355X: the sparse-MHSA kernels against dense attention.

    python bench_density.py [--L 1024] [--B 4] [--H 16] [--d 64] [--reps 20]

Follows the run-time study and the span-specialisation ablation of the
paper's evaluation (section 10): run time of the sparse primitives against
mask density for windowed, blocked and strided masks at L = 1024, densities
0.4% .. 100%.  Every point is timed on synthetic bf16 inputs resident on the
GPU.  A measurement captures `reps` back-to-back calls into one HIP graph,
times its replay with hipEvents (median of 5 replays) and divides by `reps`,
so the host cost of a call drops out; the fused forward is also timed as
eager calls, host cost included.  Per point:

* the fused forward (splat_sparse_mhsa_fwd),
* the unfused chain (splat_rsddmm, splat_row_softmax, splat_rspmm), each step,
* R-SpMM, R-SDDMM and the fused forward on a plan without span
  specialisation (SPLAT_PLAN_NO_SPAN: every row group walks all of [0, L)),
* the data-layout comparison: the transpose to the column-compressed,
  column-major layout and R-SpMM reading it, against R-SpMM on the
  row-major values the softmax leaves (masks whose columns are single
  affine runs; the paper's switch takes the column-major layout from 10%),
* dense references on the same GPU: torch.matmul (hipBLASLt) for the dense
  products Q K^T and P V that a dense-library chain computes in place of
  R-SDDMM and R-SpMM, and torch's scaled_dot_product_attention with the mask
  as an additive bias (memory-efficient backend: the same result as the
  sparse path) and without a mask (flash backend: all L^2 scores).  Each
  backend is forced; one that is not available prints null.

Prints one JSON line per point and a Markdown table at the end.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import statistics
import sys

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

# (kind, params) per family, chosen so that at L = 1024 the densities land on
# the paper's grid 0.4, 0.8, 1.6, 3, 6, 12, 24, 44, 75, 100 %.
SWEEP = {
    # |i - j| <= w
    "window": [("window", {"w": w}) for w in (2, 4, 8, 16, 32, 64, 128, 256, 512, 1023)],
    # own block and the one before it
    "blocked": [("blocked", {"block": b}) for b in (2, 4, 8, 16, 32, 64, 128, 256, 512, 1024)],
    # causal local window plus every stride-th column; causal, so at most about 50%
    "strided": [("strided_local", {"local": n, "stride": s})
                for n, s in ((4, 1024), (8, 1024), (16, 512), (24, 64), (32, 16), (128, 128),
                             (256, 16), (640, 8))],
}


def timed(fn, reps: int) -> float:
    """Median over 5 batches of `reps` eager calls of the per-call time in µs
    (includes the host cost of each call when that exceeds the kernel's)."""
    import torch
    for _ in range(3):
        fn()
    torch.cuda.synchronize()
    out = []
    for _ in range(5):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        out.append(e0.elapsed_time(e1) / reps * 1e3)
    return statistics.median(out)


def graph_timed(fn, reps: int) -> float:
    """As `timed`, but the `reps` calls are captured once into a HIP graph and
    the graph is replayed: the per-call host cost drops out, the launches stay."""
    import torch
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for _ in range(3):
            fn()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for _ in range(reps):
            fn()
    return timed(g.replay, 1) / reps


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--L", type=int, default=1024)
    ap.add_argument("--B", type=int, default=4)
    ap.add_argument("--H", type=int, default=16)
    ap.add_argument("--d", type=int, default=64)
    ap.add_argument("--reps", type=int, default=20)
    ap.add_argument("--families", default=",".join(SWEEP))
    args = ap.parse_args()

    import numpy as np
    import torch
    import torch.nn.functional as F
    from torch.nn.attention import SDPBackend, sdpa_kernel
    import paper_2407_16847_amd as splat
    import workloads

    if not torch.cuda.is_available():
        print("bench_density.py needs a GPU", file=sys.stderr)
        return 1
    L, B, H, d = args.L, args.B, args.H, args.d
    w = workloads.Workload("density_sweep", B, H, L, d, "bf16", workloads.make_pattern("full"),
                           1.0, 17)
    Q, K, V = (x.cuda() for x in workloads.make_qkv(w))
    Kt = K.transpose(-1, -2).contiguous()      # dense Q K^T takes a contiguous right operand
    scale = 1.0 / math.sqrt(d)
    O = torch.empty_like(Q)

    def dense_time(run, what):
        """Graph-replay time of a torch call, eager if it cannot be captured, None if it fails."""
        try:
            run()
            torch.cuda.synchronize()
        except RuntimeError as e:
            print(f"# {what}: unavailable ({str(e).splitlines()[0][:120]})", flush=True)
            return None
        try:
            return graph_timed(run, args.reps)
        except RuntimeError as e:
            print(f"# {what}: timed eagerly ({str(e).splitlines()[0][:120]})", flush=True)
            torch.cuda.synchronize()
            return timed(run, args.reps)

    def sdpa(backend, bias=None):
        def run():
            with sdpa_kernel([backend]):
                return F.scaled_dot_product_attention(Q, K, V, attn_mask=bias, scale=scale)
        return dense_time(run, str(backend))

    # bring the GPU to its steady clock before anything is timed (untimed)
    from bench import settle
    full = splat.Acsr(splat.Pattern.full(L))
    settle(lambda: splat.sparse_mhsa_fwd(full, Q, K, V, scale, O=O), 300.0)
    full.close()
    Pd = torch.softmax(torch.matmul(Q, Kt).float() * scale, dim=-1).to(torch.bfloat16)
    dense = {"flash_us": sdpa(SDPBackend.FLASH_ATTENTION),
             "qk_matmul_us": dense_time(lambda: torch.matmul(Q, Kt), "matmul Q K^T"),
             "pv_matmul_us": dense_time(lambda: torch.matmul(Pd, V), "matmul P V")}
    print(json.dumps({"dense": dense, "B": B, "H": H, "L": L, "d": d}), flush=True)

    def r(x):
        return None if x is None else round(x, 2)

    rows = []
    for fam in args.families.split(","):
        for kind, params in SWEEP[fam]:
            p = {k: min(v, L - 1 if k == "w" else L) for k, v in params.items()}
            pat = splat.Pattern.named(kind, p, L)
            a = splat.Acsr(pat)
            nnz = a.nnz
            S = torch.empty((B, H, nnz), dtype=torch.float32, device="cuda")
            P = torch.empty_like(S)
            t = {
                "fused": graph_timed(lambda: splat.sparse_mhsa_fwd(a, Q, K, V, scale, O=O), args.reps),
                "rsddmm": graph_timed(lambda: splat.rsddmm(a, Q, K, scale, S=S), args.reps),
                "softmax": graph_timed(lambda: splat.row_softmax(a, S, P), args.reps),
                "rspmm": graph_timed(lambda: splat.rspmm(a, P, V, O=O), args.reps),
                "fused_eager": timed(lambda: splat.sparse_mhsa_fwd(a, Q, K, V, scale, O=O),
                                     args.reps),
            }
            ac = splat.Acsr(pat, columns=True)
            if ac.info()["columns"] == 1:
                Pt = torch.empty_like(P)
                t["transpose"] = graph_timed(lambda: splat.transpose_colmajor(ac, P, Pt), args.reps)
                t["rspmm_colmajor"] = graph_timed(lambda: splat.rspmm_colmajor(ac, Pt, V, O=O),
                                                  args.reps)
                del Pt
            else:
                t["transpose"] = t["rspmm_colmajor"] = None
            ac.close()
            ns = splat.Acsr(pat, span=False)
            t["rspmm_nospan"] = graph_timed(lambda: splat.rspmm(ns, P, V, O=O), args.reps)
            t["rsddmm_nospan"] = graph_timed(lambda: splat.rsddmm(ns, Q, K, scale, S=S), args.reps)
            t["fused_nospan"] = graph_timed(lambda: splat.sparse_mhsa_fwd(ns, Q, K, V, scale, O=O),
                                            args.reps)
            rp, ci = a.export()
            rows_idx = np.repeat(np.arange(L), np.diff(rp))
            bias = torch.full((L, L), float("-inf"), dtype=torch.bfloat16)
            bias[torch.from_numpy(rows_idx).long(), torch.from_numpy(ci).long()] = 0
            t["dense_masked"] = sdpa(SDPBackend.EFFICIENT_ATTENTION, bias.cuda())
            flops = 4.0 * nnz * d * B * H
            row = {"family": fam, "kind": kind, "params": p, "density": nnz / (L * L),
                   "fused_TFLOPs": round(flops / t["fused"] / 1e6, 1),
                   "unfused_us": r(t["rsddmm"] + t["softmax"] + t["rspmm"]),
                   "span_speedup_rspmm": round(t["rspmm_nospan"] / t["rspmm"], 2),
                   "switch_picks_colmajor": bool(t["transpose"] is not None
                                                 and nnz / (L * L) >= splat.DENSE_ALPHA),
                   **{f"{k}_us": r(v) for k, v in t.items()},
                   **{f"dense_{k}": r(v) for k, v in dense.items()}}
            rows.append(row)
            print(json.dumps(row), flush=True)
            del S, P
            a.close()
            ns.close()

    def f(x):
        return "null" if x is None else f"{x:g}"

    print("\n| family | params | density | fused µs | fused TFLOP/s | fused eager µs | "
          "R-SDDMM µs | softmax µs | R-SpMM µs | R-SpMM no span µs | span speedup | "
          "fused no span µs | transpose + col-major R-SpMM µs | dense masked SDPA µs |")
    print("|---|---|---|---|---|---|---|---|---|---|---|---|---|---|")
    for x in rows:
        ps = ",".join(f"{k}={v}" for k, v in x["params"].items())
        print(f"| {x['family']} | {ps} | {100 * x['density']:.2f}% | {f(x['fused_us'])} | "
              f"{f(x['fused_TFLOPs'])} | {f(x['fused_eager_us'])} | {f(x['rsddmm_us'])} | "
              f"{f(x['softmax_us'])} | {f(x['rspmm_us'])} | {f(x['rspmm_nospan_us'])} | "
              f"{f(x['span_speedup_rspmm'])} | {f(x['fused_nospan_us'])} | "
              f"{f(x['transpose_us'])} + {f(x['rspmm_colmajor_us'])} | "
              f"{f(x['dense_masked_us'])} |")
    print(f"\ndense, independent of the mask: flash SDPA {f(r(dense['flash_us']))} µs, "
          f"matmul Q K^T {f(r(dense['qk_matmul_us']))} µs, "
          f"matmul P V {f(r(dense['pv_matmul_us']))} µs")
    return 0


if __name__ == "__main__":
    sys.exit(main())
