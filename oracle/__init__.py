"""Plain, slow, fp64 CPU oracle for the COBS decode-step path.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import anything from this package.  The
product path (the HIP library and its Python binding) never imports, links or
executes it, and this package imports nothing from the product path.

Every function states the passage of the paper (COBS: Cumulant Order Block
Sparse Attention) it writes out.  Arithmetic is float64 unless the passage fixes
a storage precision (bf16 / fp32 / FP4 E2M1 descriptor storage), in which case
the rounding is written out explicitly.

Modules
-------
``numerics``  bf16 / fp32 rounding and the FP4 E2M1 codec (Sec. 5.5).
``records``   the per-block descriptor record byte layout (Sec. 5.3, 5.5).
``method``    block statistics, log-mass estimate, GQA group score, top-s
              selection, union and sparse attention, exact-mass diagnostics
              (Sec. 2, 3, 4, 5).
``traffic``   KV-cache read-traffic accounting (Table "bandwidth", Table "quant").

Pinning status
--------------
All of ``method`` and ``traffic`` are pinned by tests under ``tests/`` against
closed forms, identities, brute force and the paper's printed tables.  The FP4
codec is pinned to the E2M1 value grid, round-to-nearest-even and the paper's
byte counts; the choice of scale (max|x|/6, one fp32 scale per vector) is a
reading of a passage that does not fix it, so that one convention is
"parity unpinned" beyond the byte counts.
"""

from . import numerics, records, method, traffic  # noqa: F401
