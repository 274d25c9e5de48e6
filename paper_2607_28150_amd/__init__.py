"""MI355X-native selective KV-cache transfer hot path (SmartGen, arXiv 2607.28150).

The work runs in libsmartgen.so (HIP kernels for gfx950 behind the C ABI of
include/smartgen.h); ``smartgen`` is its ctypes binding.
"""
from . import smartgen  # noqa: F401
