"""SparsePR sparse attention operator for AMD Instinct MI355X (gfx950).

The operator runs in the HIP library libsparsepr.so (C ABI in
include/sparsepr.h); `sparsepr` is its ctypes binding and `workloads` the
seeded synthetic input generator.  Nothing is loaded at import time.
"""
__all__ = ["sparsepr", "workloads"]
