"""MI355X (gfx950) implementation of the SPDP collapsed-Gibbs sweep.

The compute path is libspdp.so (hand-written HIP kernels behind the C ABI of
include/spdp.h); ``spdp`` is its ctypes binding.
"""
from . import spdp  # noqa: F401
