"""MI355X-native verification step of distributed speculative inference.

The package is the HIP library libdsi.so (kernels and C ABI in csrc/, header
include/dsi.h) plus a ctypes binding with the same function names (dsi.py)
and a weight-upload helper (loader.py).
"""
from . import dsi
from .dsi import DsiError, load

__all__ = ["dsi", "DsiError", "load"]
