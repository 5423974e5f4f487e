"""MI355X evaluator of candidate collective schedules (TACCL, arXiv 2111.04867).

The work runs in libtaccl.so (HIP kernels for gfx950 behind the C ABI of
include/taccl.h); `binding` is its thin ctypes binding.
"""
__all__ = ["binding"]
