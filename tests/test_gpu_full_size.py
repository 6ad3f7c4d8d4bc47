"""The decode workloads at their full sizes, through the calls and per-step
length bounds the benchmark times, against the oracle by the step protocol of
tests/protocol.py (re-synced from the GPU's pre-step state every step; no
unit dropped):

  * 8B layer H2O (64 requests x 8 KV heads, 32768-token contexts, B = 2048):
    every unit, 8 steps.  Step 1 reads 32769 slots per unit (three
    work-groups per unit, the combine kernel, then the general eviction
    kernel, 32769 -> 2048); later steps are the one-launch steady step
    (finish_steady, 512 threads).
  * 8B layer Quest (32 requests x 8 KV heads, 2048 pages, top-64): every unit,
    8 steps of the one-launch se_decode_step_quest (bounds, top-k and
    attention in one 1024-thread work-group per unit).
  * Ragged continuous batch (128 requests x 8 KV heads, retained 1024..4096,
    B = 4096): every unit, 8 steps; the longest units evict every step
    (finish_steady_strided), the others grow.
  * 32-layer loop (256 requests x 8 KV heads x 32 layers, B = 4096, ~137 GB of
    KV): 64 seeded (layer, unit) samples, 8 steps of all 32 layers
    (finish_steady_strided, 512 threads).

Inputs are generated on the device by the seeded generators.
"""
import pytest
import torch

from tests.protocol import h2o_trajectory, quest_trajectory
from workloads import LAYER_H2O, LAYER_QUEST, MODEL_H2O, RAGGED_H2O, build_state, build_steps, step_bounds

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
N_STEPS = 8


@pytest.fixture(scope="module")
def se():
    import paper_2609_39068_amd as m
    assert torch.cuda.is_available()
    return m


def _sample(w, n, seed):
    g = torch.Generator().manual_seed(seed)
    picks = set()
    while len(picks) < n:
        layer = int(torch.randint(0, w.layers, (1,), generator=g))
        unit = int(torch.randint(0, w.units_per_layer, (1,), generator=g))
        picks.add((layer, unit))
    check = {}
    for layer, unit in sorted(picks):
        check.setdefault(layer, []).append(unit)
    return check


def _h2o(se, w, check=None):
    print(f"generating {w.name}", flush=True)
    gs = build_state(w, DEV)
    steps = build_steps(w, gs, DEV, steps=N_STEPS)
    bounds = step_bounds(w, gs.lengths.cpu().tolist(), N_STEPS)
    if check is None:
        check = {l: range(w.units_per_layer) for l in range(w.layers)}
    n, near = h2o_trajectory(se, gs, steps, N_STEPS, check, q_per_kv=w.q_per_kv, scale=w.scale, budget=w.budget,
                             recent=w.recent, bounds=bounds, device=DEV)
    print(f"{n} unit-steps checked, {near} with a near-tie float64 retention", flush=True)
    return n


@pytest.mark.timeout(600)
def test_8b_layer_h2o_full_size(se):
    w = LAYER_H2O
    assert _h2o(se, w) == N_STEPS * w.units_per_layer


@pytest.mark.timeout(600)
def test_ragged_batch_h2o_full_size(se):
    w = RAGGED_H2O
    assert _h2o(se, w) == N_STEPS * w.units_per_layer


@pytest.mark.timeout(600)
def test_32_layer_h2o_full_size(se):
    w = MODEL_H2O
    check = _sample(w, 64, seed=w.seed + 99)
    assert _h2o(se, w, check) == N_STEPS * 64


@pytest.mark.timeout(600)
def test_8b_layer_quest_full_size(se):
    w = LAYER_QUEST
    print(f"generating {w.name}", flush=True)
    gs = build_state(w, DEV)
    steps = build_steps(w, gs, DEV, steps=N_STEPS)
    bounds = step_bounds(w, gs.lengths.cpu().tolist(), N_STEPS)
    n, near = quest_trajectory(se, gs, steps, N_STEPS, range(w.units_per_layer), q_per_kv=w.q_per_kv,
                               scale=w.scale, top_k=w.top_k, bounds=bounds, device=DEV)
    print(f"{n} unit-steps checked, {near} with a near-tie float64 selection", flush=True)
    assert n == N_STEPS * w.units_per_layer
