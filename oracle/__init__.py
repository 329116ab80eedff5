"""CPU fp64 oracle for the Dion2 step. Test infrastructure only: imported by
tests, the smoke check and the benchmark's CPU-baseline leg, never by the
product path."""
from .dion2_oracle import *  # noqa: F401,F403
from .dion2_oracle import (AXIS_AUTO, AXIS_COLS, AXIS_ROWS, DEFAULT_EPS,  # noqa: F401
                           DEFAULT_LR, DEFAULT_MU, MUON_QUINTIC)
