"""MI355X-native grid coevolution of GANs (Lipizzaner, arXiv 1811.12843).

The compute path is liblipz.so (HIP kernels for gfx950 behind the C ABI in
include/lipz.h); this package is its thin ctypes binding.  PyTorch is used by
callers only to allocate device memory and obtain streams.
"""
from .lipz import *  # noqa: F401,F403
