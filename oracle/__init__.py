"""CPU oracle for Grouped Cross Attention -- TEST INFRASTRUCTURE ONLY.

Plain fp64 numpy, written from the paper's equations.  Only ``tests/``, the
smoke check in ``__graft_entry__`` and the benchmark's CPU-baseline leg may
import anything from this package.  It never imports the GPU package and the
GPU package never imports it.
"""

from . import gca  # noqa: F401
