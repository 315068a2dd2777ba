"""fp64 CPU oracle for the ragged paged attention path (test infrastructure only).

Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg may import
this package.  The product library never imports it and shares no code with it.
"""
from .tangram import *  # noqa: F401,F403
from .tangram import (MODE_AOT, MODE_NAIVE, MODE_UNIFORM, MODE_FILL, MODE_SPLIT_MAP, GROUP_CLUSTERED, GROUP_ADJACENT,  # noqa: F401
                      OracleError, OutOfPages)
