"""Dion2 optimizer step for AMD Instinct MI355X (gfx950).

The step runs in libdion2.so (hand-written HIP kernels behind a C ABI,
include/dion2.h); `binding` marshals torch tensors into it and `workloads`
builds seeded synthetic optimizer states shaped like the paper's models.
"""
from . import binding  # noqa: F401
from .binding import (AXIS_AUTO, AXIS_COLS, AXIS_ROWS, Dion2Error,  # noqa: F401
                      dion2_last_error, dion2_plan_info, dion2_release_workspaces,
                      dion2_status_string, dion2_step, dion2_step_batched, dion2_step_ex,
                      dion2_step_strided, dion2_version, dion2_workspace_size)
