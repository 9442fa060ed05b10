"""Seeded synthetic inputs for Grouped Cross Attention workloads.

This package is shared by the GPU path's tests and benchmark and by the CPU
oracle's tests.  It draws random numbers and lays them out; it holds none of
the method's arithmetic (no scores, no selection, no attention).  Anything
that needs a landmark score, such as the top-k margin check, lives with the
oracle and calls back into :func:`gen.inputs.redraw_lmk_q_row`.
"""

from .workloads import WORKLOADS, Workload, get_workload  # noqa: F401
from . import bf16, inputs  # noqa: F401
