"""MI355X-native candidate ranking over a shared user-history KV cache.

The compute lives in libupr.so (HIP kernels for gfx950 behind the C interface
of include/upr.h); ``paper_2606_00422_amd.upr`` is its ctypes binding.
"""
from . import upr  # noqa: F401

__all__ = ["upr"]
