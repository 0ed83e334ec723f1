"""Reference oracle for sparse multi-head self-attention over regular masks.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this package: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code with the HIP
path (``paper_2407_16847_amd``) and imports nothing from it; the only module
both sides use is ``workloads`` (seeded input generation, no method
arithmetic).

What it computes, plainly and slowly, in fp64 on the CPU:

* ``masks``     -- the attention mask of every workload pattern, enumerated by
                   brute force over all (i, j) from the pattern's defining
                   predicate; the CSR view (row_ptr, col_idx) of that mask is
                   the reference ACSR index set (section 4.1, point-sets).
* ``acsr``      -- the paper's ACSR definitions: affine-compressibility
                   (section 4.1, Definition 1), the two-point affine-index solve
                   and the regularity check (section 5.1), the sparse-to-dense
                   column map (section 5.1) and O(1) membership ("fast
                   indexing", section 5.2).
* ``attention`` -- masked attention, Equation 1 with the softmax taken over
                   each row's non-zeros only: S = scale * Q K^T on the mask,
                   P = row softmax of S, O = P V; dense per head, plus a
                   per-row variant for sampled rows at full size.

Every function is pinned by ``tests/test_oracle_*.py`` against values fixed
by the paper or by mathematics (worked examples, closed forms, invariants,
special cases that reduce to library routines, brute force on tiny inputs).
"""
from . import acsr, attention, masks  # noqa: F401
