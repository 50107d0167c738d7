"""Spatially-sparse DeepCNet (arXiv:1409.6070) forward and backward pass on AMD MI355X.

The computation lives in ``libsscn.so`` (HIP kernels for gfx950 behind the C
interface in ``include/sscn.h``); ``sscn`` is its ctypes binding.
"""

__all__ = ["sscn"]
