"""SANTA / S2ANTA decode-step attention for AMD Instinct MI355X (gfx950).

The compute path is libsanta.so (hand-written HIP kernels behind a C ABI,
include/santa.h); ``paper_2605_01910_amd.santa`` is its ctypes binding.
"""

from . import santa  # noqa: F401
