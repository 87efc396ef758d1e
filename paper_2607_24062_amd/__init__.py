"""MI355X (gfx950) scoring and discrepancy path of ACRL.

The computation lives in libacrl.so (HIP kernels behind the C ABI of
include/acrl.h); ``paper_2607_24062_amd.acrl`` is its ctypes binding.
"""
from . import acrl  # noqa: F401

__all__ = ["acrl"]
