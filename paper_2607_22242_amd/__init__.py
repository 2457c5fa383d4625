"""Brute-force device-mapping search on MI355X (HIP for gfx950).

The search itself lives in libsched.so (C ABI declared in
include/sched_search.h); `binding` marshals arguments to it.
"""
from .binding import (  # noqa: F401
    EXPORTED, INFEASIBLE, NO_INDEX, Monitor, Problem, SchedError, sched_bruteforce_argmin,
    sched_bruteforce_argmin_noalloc, sched_bruteforce_record,
    sched_eval_batch, sched_eval_mappings, sched_eval_mappings_device, sched_eval_reprobes,
    sched_num_mappings, sched_num_tools,
    sched_mapping_index, sched_mapping_modes, sched_problem_create, sched_problem_create_desc,
    sched_problem_create_masked,
    sched_monitor_averages, sched_monitor_create, sched_monitor_destroy, sched_monitor_latencies,
    sched_monitor_observe, sched_problem_destroy, sched_pruned_argmin,
    sched_pruned_workspace_bytes, pruned_workspace, sched_strerror, sched_valu_probe,
    sched_wave_or_probe, sched_workspace_bytes, workspace)
