"""fp4root: NVFP4 Newton-Schulz orthogonalisation (the paper's Q-Root) on AMD gfx950.

The compute lives in ``libfp4root.so`` (hand-written HIP kernels behind a C
ABI declared in ``include/fp4root.h``); ``paper_2607_04422_amd.fp4root`` is a
thin ctypes binding with the same entry-point names.  Importing this package
loads nothing; the library is loaded on first use and a missing library is an
error, never a fallback.
"""

__all__ = ["fp4root", "workloads", "build"]
