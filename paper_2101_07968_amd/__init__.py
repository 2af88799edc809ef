"""DynaComm's segment-overlapped parameter-server iteration on MI355X.

The work happens in libdc.so (HIP kernels for gfx950, the planner and the
executor behind the C ABI of include/dc.h); this package is its ctypes
binding plus the workload definitions.
"""
from ._lib import (DC_OPT_LR, DC_OPT_SGD_THREADS, DC_OPT_TIMELINE, DC_OPT_TIMEOUT_S, DcError, Model, Plan,  # noqa
                   Profile, dc_plan, dc_plan_eval, dc_plan_lbl, dc_plan_sequential, lib, link)
from . import nets  # noqa: F401
