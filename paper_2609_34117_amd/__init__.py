"""SlimWise batched-decode MoE layer for MI355X (gfx950).

The compute lives in ``libslimwise.so`` (hand-written HIP kernels behind a C
ABI declared in ``include/slimwise.h``).  ``paper_2609_34117_amd.slimwise``
is the thin ctypes binding with the same call names; ``inputs`` draws the
seeded synthetic workloads.  Importing the package does not load the HIP
library; the binding does, and raises if it is missing.
"""

__all__ = ["inputs", "slimwise"]
