"""MI355X (gfx950) speculate-reuse-repair decode path for dynamic sparse attention.

The compute lives in libprr.so (hand-written HIP kernels behind the C ABI of
include/prr.h); this package is its ctypes binding plus a thin two-stream runtime.
"""
from ._lib import *  # noqa: F401,F403
from ._lib import EXPORTED, PrrError, library, make_dims  # noqa: F401
