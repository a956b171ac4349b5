"""Seeded synthetic inputs for the ALP allocation search (shared by the oracle side and the GPU side)."""
from .alp_workloads import (  # noqa: F401
    CONFIGS,
    WorkloadConfig,
    make_instance,
    make_batch,
    make_custom,
    num_options,
    num_candidates,
    sample_indices,
    target_from_tmax,
)
