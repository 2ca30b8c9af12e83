"""HySparse2 hybrid-block decode attention for MI355X (gfx950).

The compute lives in ``libhs2.so`` (hand-written HIP kernels behind a C ABI,
declared in include/hs2.h).  ``paper_2609_26368_amd.hs2`` is its thin ctypes
binding; ``paper_2609_26368_amd.workloads`` draws seeded synthetic inputs.
Importing the package loads nothing: the library is opened on first use and
raises if it has not been built.
"""
__all__ = ["hs2", "workloads"]
