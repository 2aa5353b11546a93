"""MI355X-native sparse absorbed-MLA partial attention and LSE merge.

The compute lives in a HIP/C++ shared library (`libmla_sparse.so`, C ABI
declared in `include/mla_sparse.h`); `paper_2606_01502_amd.mla` is the thin
Python binding over it.  Importing this package loads nothing; the library
is loaded on first use of the binding.
"""
__all__ = ["mla", "workloads"]
