"""Seeded synthetic workload generators (no pruning arithmetic)."""

from .workloads import (WORKLOADS, DEFAULT_BENCH_WORKLOAD, Workload,  # noqa: F401
                        keep_count, sensitivity_inputs, stage1_inputs, stage2_inputs, sweep,
                        to_storage)
