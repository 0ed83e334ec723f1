#!/usr/bin/env python3
"""Thread-block counts of three tilings of the paper's masks (host only).

    python bench_tiling.py [--L 1024] [--out FILE]

The SDDMM tiling ablation of the paper's evaluation (section 10) counts the
thread-blocks poset tiling (section 7.3) needs against a naive tiling, for
windowed and blocked masks at L = 1024 over their densities.  Here, per mask
of the density grid (the same families and parameters as bench_density.py):

* poset tiling and the grid arrangement (unstretched blocks at every multiple
  of the block shape that meet the mask) with 16 x 16 blocks, the shape the
  paper's reported thread savings divide into, and with the 32 x 64
  wavefront tile of this library's kernels;
* this library's own plan: its wavefront-tiles (32 rows x 64 keys) that hold
  at least one key, and the share of their computed points in the mask.

Writes a Markdown table (stdout, or --out).  No GPU is used.
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


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--L", type=int, default=1024)
    ap.add_argument("--out", default=None)
    args = ap.parse_args()
    import paper_2407_16847_amd as splat

    L = args.L
    lines = [f"# Thread-block counts of poset, grid and row-group tilings, L = {L}", "",
             "Command (from the repository root, host only):", "", "```",
             "python bench_tiling.py" + (f" --L {L}" if L != 1024 else ""), "```", "",
             "λ is the number of thread-blocks; grid/poset is the reduction poset tiling "
             "achieves over the grid arrangement; saved = (λ_grid − λ_poset) × threads per block. "
             "Stretch: the one poset tiling selects (section 7.3.1). Plan: this library's "
             "non-empty 32 × 64 wavefront-tiles and nnz / computed points.", "",
             "| family | params | density | λ poset 16×16 | λ grid 16×16 | grid/poset | saved threads "
             "| stretch | λ poset 32×64 | λ grid 32×64 | plan tiles 32×64 | plan efficiency |",
             "|---|---|---|---|---|---|---|---|---|---|---|---|"]
    ratios = {}
    for fam, pats in list(SWEEP.items()) + list(EXTRA.items()):
        for kind, params in pats:
            p = {k: min(v, L - 1 if k == "w" else L) for k, v in params.items()}
            a = splat.Acsr(splat.Pattern.named(kind, p, L))
            info = a.info()
            ps = a.tiling("poset", 16, 16)
            gs = a.tiling("grid", 16, 16)
            pw = a.tiling("poset", 32, 64)
            gw = a.tiling("grid", 32, 64)
            plan_tiles = info["computed"] // (32 * 64)
            r = gs["blocks"] / ps["blocks"]
            ratios.setdefault(fam, []).append(r)
            lines.append(
                f"| {fam} | {','.join(f'{k}={v}' for k, v in p.items())} | "
                f"{100 * info['nnz'] / L ** 2:.2f}% | {ps['blocks']} | {gs['blocks']} | {r:.3f} | "
                f"{(gs['blocks'] - ps['blocks']) * 256} | {ps['stretch']} | {pw['blocks']} | "
                f"{gw['blocks']} | {plan_tiles} | {info['nnz'] / info['computed']:.3f} |")
            a.close()
    lines += ["", "Reduction of the thread-block count by poset tiling over the grid arrangement "
              "(16 × 16 blocks):", "", "| family | mean | geomean | max |", "|---|---|---|---|"]
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
