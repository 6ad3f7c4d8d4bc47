"""Seeded synthetic workloads (sizes and random inputs only; no method arithmetic)."""
from .configs import (CONFIGS, H2O_PREFILL, LAYER_H2O, LAYER_QUEST, MODEL_H2O, OMNIKV, PRUNE,  # noqa: F401
                      RAGGED_H2O, SNAPKV, TINY_H2O, Workload, scaled, step_bounds)
from .generate import (  # noqa: F401
    PagedInputs, StepInputs, build_observation, build_state, build_steps, clone_state, heavy_hitter, isolated_units, observation_queries,
    to_device,
    unit_slots)
