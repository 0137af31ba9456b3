"""MI355X (gfx950) library for FOVEA's per-draft-step visual-evidence retrieval and fusion.

The computation lives in ``lib/libfovea.so`` (hand-written HIP kernels behind the C ABI
of ``include/fovea.h``); ``fovea`` is its ctypes binding.
"""

from .fovea import *  # noqa: F401,F403
from .fovea import Fovea, FoveaError, Outputs  # noqa: F401
