"""Seeded synthetic workloads (sizes and random inputs only; no method arithmetic)."""
from .configs import CONFIGS, Workload, scaled  # noqa: F401
from .generate import (  # noqa: F401
    PagedInputs, StepInputs, build_state, build_steps, clone_state, heavy_hitter, isolated_units, to_device,
    unit_slots)
