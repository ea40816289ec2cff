"""MI355X (gfx950) hot path of SparOA (arXiv 2511.19457).

The compute lives in libsparoa.so (hand-written HIP kernels behind a C ABI,
declared in include/sparoa.h); ``abi`` is its ctypes binding and ``driver``
the per-layer measure -> route -> execute loop over network-shaped stacks.
"""
from . import abi  # noqa: F401  (loads libsparoa.so; raises if it is not built)
from .abi import *  # noqa: F401,F403
