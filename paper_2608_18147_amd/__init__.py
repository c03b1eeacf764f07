"""MI355X (gfx950) implementation of the ECASQ approximate-DP hot path
(arXiv 2608.18147): HIP kernels behind the C ABI of include/ecasq.h, with a
thin ctypes binding in paper_2608_18147_amd.ecasq.

Importing the package loads nothing; the library is loaded on first use and
the binding raises if libecasq.so is absent.
"""
__all__ = ["ecasq", "inputs", "build"]
