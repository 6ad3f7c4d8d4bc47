"""Seeded synthetic workloads (sizes and random inputs only; no method arithmetic)."""
from .configs import CONFIGS, H2O_PREFILL, OMNIKV, PRUNE, SNAPKV, Workload, scaled  # noqa: F401
from .generate import (  # noqa: F401
    PagedInputs, StepInputs, build_observation, build_state, build_steps, clone_state, heavy_hitter, isolated_units, observation_queries,
    to_device,
    unit_slots)
