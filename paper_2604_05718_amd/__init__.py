"""Mutual Pair Merging (MPM) token reduction on MI355X (gfx950).

The computation lives in libmpm.so (hand-written HIP kernels behind the C ABI
of include/mpm.h); this package is its thin torch binding.
"""
from .api import (Merged, Schedule, ScheduleResult, affinity, affinity_schedule_used, argmax, compose,
                  compose_unmerge, insertion, local_block_rows, merge, merge_local, new_workspace, pair_average,
                  pair_compact, run_schedule, unmerge, workspace_bytes)
from ._lib import MPMError

__all__ = ["Merged", "Schedule", "ScheduleResult", "MPMError", "affinity", "affinity_schedule_used", "argmax",
           "compose", "compose_unmerge", "insertion", "local_block_rows", "merge", "merge_local", "new_workspace",
           "pair_average", "pair_compact", "run_schedule", "unmerge", "workspace_bytes"]
