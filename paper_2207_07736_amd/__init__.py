"""GPU-vectorised, kernel-fused cart-pole data collection for MI355X (gfx950).

The compute path is librlsim.so (hand-written HIP kernels behind the C ABI of
include/rlsim.h); ``rlsim`` is its thin ctypes binding.  Importing this package
loads the library and fails if it has not been built.
"""
from .rlsim import *  # noqa: F401,F403
from .rlsim import EXPORTS, LIB_PATH, RlsimError, Simulator, Trajectory, TrajRows, stats_only  # noqa: F401
