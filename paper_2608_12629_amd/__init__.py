"""Flash-KMeans Lloyd iteration for AMD Instinct MI355X (gfx950).

The compute path is ``libflashkmeans.so`` (hand-written HIP kernels behind the
C ABI declared in ``include/flashkmeans.h``); ``paper_2608_12629_amd.kmeans``
is the thin ctypes binding over it.  ``paper_2608_12629_amd.synth`` makes the
seeded synthetic workloads.  Importing this package loads nothing.
"""
__all__ = ["kmeans", "synth"]
