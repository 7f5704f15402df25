"""MI355X-native generation-stage policy forward (VLA rollout) for gfx950.

The compute lives in libebrl.so (hand-written HIP kernels behind the C ABI
of include/ebrl.h); ``paper_2609_27547_amd.ebrl`` is its ctypes binding.
"""
from . import ebrl  # noqa: F401
