#!/usr/bin/env python3
"""Thread-block counts of poset tiling against the paper's Naive Tiling
(host only).

    python bench_tiling.py [--L 1024] [--out FILE] [--step 1]

The SDDMM tiling ablation of the paper's evaluation (section 10) counts the
thread-blocks poset tiling (section 7.3, Algorithm 1) needs against Naive
Tiling (Appendix C: m-row patches, each tiled left to right from its leftmost
point) for windowed and blocked masks at L = 1024 over every density the
pattern allows, and reports the mean and the largest reduction with the
threads it saves.  The paper does not print its block shape; its thread
savings are whole multiples of 256, so three 256-thread shapes are swept
(m rows x n columns: 16 x 16, 32 x 8, 64 x 4).

Part 1 sweeps every window half-width w = 0 .. L-1 and every block size
b = 1 .. L.  Part 2 is the density grid of the paper's run-time study (the
masks of bench_density.py) with, per mask: poset and naive counts at
16 x 16, the grid arrangement (unstretched blocks at every multiple of the
block shape that meet the mask, a separately labelled third tiling), the
counts at the 32 x 64 wavefront tile of this library's kernels, and this
library's own plan (its non-empty 32-row x 64-key wavefront-tiles and
nnz / computed points).

Writes Markdown (stdout, or --out).  No GPU is used.
"""
from __future__ import annotations

import argparse
import math
import os
import sys

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from bench_density import SWEEP  # noqa: E402  (the same masks as the density sweep)

EXTRA = {"dilated": [("dilated", {"w": w, "dilation": 2}) for w in (2, 8, 32, 128, 256)]}
SHAPES = [(16, 16), (32, 8), (64, 4)]
PAPER = {"window": (1.098, 1.83, 13568), "blocked": (1.095, 1.72, 12544)}


def _sweep_all(splat, L, fam, m, n, step):
    vals = range(0, L, step) if fam == "window" else range(1, L + 1, step)
    ratios, best = [], None
    for v in vals:
        pat = splat.Pattern.window(L, v) if fam == "window" else splat.Pattern.blocked(L, v)
        a = splat.Acsr(pat)
        p = a.tiling("poset", m, n, stretch=1)["blocks"]
        q = a.tiling("naive", m, n)["blocks"]
        a.close()
        r = q / p
        ratios.append(r)
        if best is None or r > best[0]:
            best = (r, v, p, q)
    return ratios, best


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--L", type=int, default=1024)
    ap.add_argument("--step", type=int, default=1, help="parameter step of part 1")
    ap.add_argument("--out", default=None)
    args = ap.parse_args()
    import paper_2407_16847_amd as splat

    L = args.L
    cmd = "python bench_tiling.py" + (f" --L {L}" if L != 1024 else "") + \
        (f" --step {args.step}" if args.step != 1 else "")
    lines = [f"# Poset tiling against Naive Tiling (Appendix C), L = {L}", "",
             "Command (from the repository root, host only):", "", "```", cmd, "```", "",
             "λ is the number of thread-blocks of m rows × n columns; naive/poset is the "
             "reduction poset tiling (stretch 1, the selection for polygonal masks) achieves "
             "over Naive Tiling; saved = (λ_naive − λ_poset) × m·n threads.", "",
             "## 1. Every density the pattern allows", "",
             f"Window half-widths w = 0 … {L - 1} and block sizes b = 1 … {L}"
             + (f" (every {args.step}th)" if args.step != 1 else "") + ". The paper's figures "
             "(section 10, SDDMM tiling) are quoted beside them.", "",
             "| family | m × n | masks | mean naive/poset | geomean | max | at | λ poset | λ naive "
             "| saved threads | paper mean | paper max | paper saved |",
             "|---|---|---|---|---|---|---|---|---|---|---|---|---|"]
    for fam in ("window", "blocked"):
        for m, n in SHAPES:
            rs, (r, v, p, q) = _sweep_all(splat, L, fam, m, n, args.step)
            g = math.exp(sum(math.log(x) for x in rs) / len(rs))
            pm, px, ps = PAPER[fam]
            lines.append(f"| {fam} | {m} × {n} | {len(rs)} | {sum(rs) / len(rs):.3f} | {g:.3f} | "
                         f"{r:.3f} | {'w' if fam == 'window' else 'b'}={v} | {p} | {q} | "
                         f"{(q - p) * m * n} | {pm} | {px} | {ps} |")
    lines += ["", "## 2. The density grid of the run-time study", "",
              "| family | params | density | λ poset 16×16 | λ naive 16×16 | naive/poset | saved "
              "threads | λ grid 16×16 | stretch | λ poset 32×64 | λ naive 32×64 | plan tiles "
              "32×64 | plan efficiency |",
              "|---|---|---|---|---|---|---|---|---|---|---|---|---|"]
    ratios = {}
    for fam, pats in list(SWEEP.items()) + list(EXTRA.items()):
        for kind, params in pats:
            p = {k: min(v, L - 1 if k == "w" else L) for k, v in params.items()}
            a = splat.Acsr(splat.Pattern.named(kind, p, L))
            info = a.info()
            ps = a.tiling("poset", 16, 16)
            ns = a.tiling("naive", 16, 16)
            gs = a.tiling("grid", 16, 16)
            pw = a.tiling("poset", 32, 64)
            nw = a.tiling("naive", 32, 64)
            plan_tiles = info["computed"] // (32 * 64)
            r = ns["blocks"] / ps["blocks"]
            ratios.setdefault(fam, []).append(r)
            lines.append(
                f"| {fam} | {','.join(f'{k}={v}' for k, v in p.items())} | "
                f"{100 * info['nnz'] / L ** 2:.2f}% | {ps['blocks']} | {ns['blocks']} | {r:.3f} | "
                f"{(ns['blocks'] - ps['blocks']) * 256} | {gs['blocks']} | {ps['stretch']} | "
                f"{pw['blocks']} | {nw['blocks']} | {plan_tiles} | {info['nnz'] / info['computed']:.3f} |")
            a.close()
    lines += ["", "Reduction of the thread-block count by poset tiling over Naive Tiling "
              "(16 × 16 blocks) on the density grid:", "", "| family | mean | geomean | max |",
              "|---|---|---|---|"]
    for fam, rs in ratios.items():
        g = math.exp(sum(math.log(x) for x in rs) / len(rs))
        lines.append(f"| {fam} | {sum(rs) / len(rs):.3f} | {g:.3f} | {max(rs):.3f} |")
    text = "\n".join(lines) + "\n"
    if args.out:
        with open(args.out, "w") as f:
            f.write(text)
    print(text, end="")
    return 0


if __name__ == "__main__":
    sys.exit(main())
