"""MoARa optimizer hot path for AMD MI355X (gfx950).

The computation lives in libmoara.so (HIP kernels behind the C ABI declared in
include/moara.h); `paper_2609_15037_amd.moara` is the ctypes binding.
"""
from . import moara  # noqa: F401
