"""Seeded synthetic inputs for the eviction step; no eviction arithmetic."""

from .workloads import (  # noqa: F401
    Workload, WORKLOADS, SWEEP_KEEP, SWEEP_RANDOM, PAPER_RANDOM_SHARE_20,
    sweep_workloads, custom, make_layer, make_grouped_layer, alg_bytes, alg_flops,
)
