"""MI355X (gfx950) implementation of Domino's per-step drafting path.

The compute lives in libdomino.so (HIP kernels behind the C ABI of
include/domino.h); `binding` is its thin ctypes binding.
"""
__all__ = ["binding", "build"]
