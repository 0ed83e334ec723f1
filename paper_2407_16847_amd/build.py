"""Build libsplat.so for gfx950 with hipcc (in-tree), and its checked twin.

    python -m paper_2407_16847_amd.build          # or __graft_entry__.build()

Every source is compiled every time (the driver's "does it build" check), the
objects in ``_build/`` and the library next to this file.  The same sources
built with -DSPLAT_DEBUG_BOUNDS give ``libsplat_checked.so`` (objects in
``_build_checked/``): every kernel checks the global-memory indices it derives
from the plan (see csrc/bounds.hpp and splat_debug_bounds in splat.h).  Its
kernels are otherwise the regular ones; it is a debugging aid, and nothing
but its own tests loads it.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
OUT = os.path.join(HERE, "libsplat.so")
BUILD_DIR = os.path.join(HERE, "_build")
OUT_CHECKED = os.path.join(HERE, "libsplat_checked.so")
BUILD_DIR_CHECKED = os.path.join(HERE, "_build_checked")
ARCH = "gfx950"

SOURCES = ["acsr_host.cpp", "tiling.cpp", "api.hip", "kernels_rows.hip", "kernels_mfma.hip", "kernels_tiles.hip"]

COMMON = ["-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-function", "-Wno-unknown-pragmas"]
# Packed fp32 instructions stay off: plain float code must not be turned into
# v_pk_* fp32 operations.
DEVICE = [f"--offload-arch={ARCH}", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-munsafe-fp-atomics"]


def hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found (ROCm is required to build libsplat.so)")


def _cmd(src: str, build_dir: str, defs: list) -> list:
    obj = os.path.join(build_dir, os.path.splitext(src)[0] + ".o")
    path = os.path.join(CSRC, src)
    if src.endswith(".hip"):
        return [hipcc(), "-x", "hip", *COMMON, *DEVICE, *defs, "-c", path, "-o", obj]
    # host-only C++ (no device code): the system C++ compiler
    return [os.environ.get("CXX", "g++"), *COMMON, *defs, "-c", path, "-o", obj]


def build(verbose: bool = False, checked: bool = False) -> str:
    """Compile and link libsplat.so (or, with ``checked``, libsplat_checked.so)."""
    target, build_dir = (OUT_CHECKED, BUILD_DIR_CHECKED) if checked else (OUT, BUILD_DIR)
    defs = ["-DSPLAT_DEBUG_BOUNDS"] if checked else []
    os.makedirs(build_dir, exist_ok=True)
    t0 = time.time()
    procs = []
    for src in SOURCES:
        cmd = _cmd(src, build_dir, defs)
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append((src, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)))
    errors = []
    for src, p in procs:
        out, _ = p.communicate()
        text = out.decode(errors="replace")
        if p.returncode != 0:
            errors.append(f"--- {src} (exit {p.returncode}) ---\n{text}")
        elif verbose and text.strip():
            print(text, flush=True)
    if errors:
        raise RuntimeError("libsplat build failed:\n" + "\n".join(errors))
    objs = [os.path.join(build_dir, os.path.splitext(s)[0] + ".o") for s in SOURCES]
    tmp = target + ".tmp"
    link = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    if verbose:
        print(" ".join(link), flush=True)
    r = subprocess.run(link, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)
    if r.returncode != 0:
        raise RuntimeError("libsplat link failed:\n" + r.stdout.decode(errors="replace"))
    os.replace(tmp, target)
    if verbose:
        print(f"built {target} in {time.time() - t0:.1f} s", flush=True)
    return target


def build_all(verbose: bool = False) -> None:
    """Both libraries: the regular one and the checked one."""
    build(verbose=verbose)
    build(verbose=verbose, checked=True)


if __name__ == "__main__":
    build_all(verbose="-q" not in sys.argv)
