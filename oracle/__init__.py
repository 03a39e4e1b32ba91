"""fp64 CPU oracle of the CommitKV hot path (test infrastructure only).

Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg import it.
"""
from .commitkv_oracle import *  # noqa: F401,F403
from .commitkv_oracle import (CANDIDATE, DORMANT, FREE, NEWLY_ACTIVE,  # noqa: F401
                              PROTECTED, RETIRED, STILL_ACTIVE, UNCERTAIN)
