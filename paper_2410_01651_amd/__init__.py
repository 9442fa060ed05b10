"""libgca: the Grouped Cross Attention hot path on MI355X (gfx950).

The compute lives in ``libgca.so`` (HIP kernels behind the C ABI declared in
``include/gca.h``); :mod:`paper_2410_01651_amd.gca` is its ctypes binding.
"""

from . import gca  # noqa: F401
from .gca import GcaError, Problem, problem  # noqa: F401
