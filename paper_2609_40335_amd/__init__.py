"""MI355X-native DP-SGD ghost-clipping hot path (libdpghost).

The computation lives in HIP kernels for gfx950 behind the C ABI declared in
include/dpghost.h; ``paper_2609_40335_amd.dpghost`` is the ctypes binding.
"""
from . import dpghost  # noqa: F401
