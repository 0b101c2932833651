"""Bitserial low-precision operators for MI355X (gfx950).

The compute lives in ``libbitserial.so`` (hand-written HIP kernels behind a
C ABI, declared in ``include/bitserial.h``).  ``paper_1810_11066_amd.bitserial``
is the thin Python binding over it; ``paper_1810_11066_amd.workloads`` draws the
seeded synthetic inputs.  Nothing is imported eagerly, so importing the package
does not touch the GPU.
"""
__all__ = ["bitserial", "workloads"]
