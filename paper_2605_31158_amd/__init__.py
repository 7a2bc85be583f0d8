"""Block selection and block-sparse attention for autoregressive chunk generation on MI355X.

The compute lives in a C-ABI HIP library (libla.so, built for gfx950); this package
holds the ctypes binding (`paper_2605_31158_amd.la`) and the seeded synthetic
workloads (`paper_2605_31158_amd.workloads`).  Importing the package loads nothing;
the library is loaded on first use and a missing library is an error.
"""
__all__ = ["la", "workloads"]
