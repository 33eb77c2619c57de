"""Batched what-if simulation of trace-derived task graphs on MI355X.

The compute path is libdd.so (HIP kernels for gfx950 behind the C-ABI of
include/dd.h); `binding` exposes it with the same names.
"""
from . import binding  # noqa: F401
from .binding import (DD_LEVELS, DD_LOAD_SHARED_THREADS, DD_PHASES,  # noqa: F401
                      DD_POLICY_EARLIEST, DD_POLICY_PRIORITY, DDError, dd_apply_transforms,
                      dd_graph_free, dd_graph_load, dd_graph_load_ex, dd_last_error,
                      dd_levelize, dd_release_cache, dd_runtime_breakdown, dd_sched_free,
                      dd_sched_info, dd_sched_task_steps, dd_simulate_batch,
                      dd_simulate_batch_noalloc, dd_simulate_batch_vs, dd_simulate_policy,
                      dd_status_str, dd_variants_free)
