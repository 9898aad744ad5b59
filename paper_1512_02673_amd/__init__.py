"""(n,k) MDS-coded matrix multiplication on one MI355X (gfx950).

The computation runs in the HIP library built from csrc/ (C ABI in
include/coded.h); `binding` exposes its calls to Python under the same names.
"""
__all__ = ["binding", "build"]
