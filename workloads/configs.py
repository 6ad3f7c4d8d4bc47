"""The five synthetic decode workloads and their scaled-down test variants.

These stand in for the paper's long-context decode benchmark (Appendix D,
"Long-Context Decode Benchmark" and "Serving Performance with 32K-token
Inputs": 128K and 32K inputs, 16-token pages, retained budgets of 2,048 and
4,096 tokens), whose models and prompts are not available.  The head shape
Hq=32, Hkv=8, d=128 is the Llama-3-8B GQA shape.

Nothing here computes any part of the method; it only names sizes.
"""

from dataclasses import dataclass, replace
from typing import Optional, Tuple


@dataclass(frozen=True)
class Workload:
    index: int
    name: str
    method: str                      # "h2o", "quest", "snapkv" (prompt compaction), "omnikv", "h2o_prefill"
                                     # or "prune" (interval prefix-cache pruning)
    num_req: int
    hq: int
    hkv: int
    head_dim: int
    layers: int
    steps: int
    page_size: int = 16
    ctx: Optional[int] = None        # initial logical context per request (uniform)
    ctx_log_range: Optional[Tuple[int, int]] = None       # log-uniform context per request
    retained_range: Optional[Tuple[int, int]] = None      # per-head retained length, uniform
    initial_resident: Optional[int] = None                # resident slots per head (< ctx)
    budget: Optional[int] = None     # H2O retained budget B
    recent: Optional[int] = None     # H2O protected recent window w
    top_k: Optional[int] = None      # Quest selected pages per KV head
    obs_window: Optional[int] = None  # SnapKV observation window w (the prompt's last w positions)
    pool_kernel: Optional[int] = None  # SnapKV max-pooling width kappa
    filter_layers: Optional[Tuple[int, ...]] = None  # OmniKV observation layers (full attention + selection)
    chunk: Optional[int] = None      # H2O prefill: the chunk's length (its queries' last obs_window score)
    interval: Optional[Tuple[int, int]] = None  # prefix pruning: the history interval [lo, hi) pruned
    hh_rate: float = 0.0             # share of positions whose key gets += hh_shift * u
    hh_shift: float = 0.0
    relevant_pages: int = 0          # Quest: pages whose keys all get += relevant_shift * u
    relevant_shift: float = 0.0
    seed: int = 0

    @property
    def q_per_kv(self) -> int:
        return self.hq // self.hkv

    @property
    def units_per_layer(self) -> int:
        return self.num_req * self.hkv

    @property
    def scale(self) -> float:
        import numpy as np
        return float(np.float32(1.0 / np.sqrt(self.head_dim)))


CONFIGS = [
    Workload(0, "tiny-h2o-step", "h2o", num_req=2, hq=8, hkv=2, head_dim=64, layers=1,
             steps=1, ctx=512, budget=128, recent=64, hh_rate=0.01, hh_shift=4.0, seed=0),
    Workload(1, "llama3-8b-layer-h2o", "h2o", num_req=64, hq=32, hkv=8, head_dim=128, layers=1,
             steps=256, ctx=32768, budget=2048, recent=256, hh_rate=0.01, hh_shift=4.0, seed=1),
    Workload(2, "llama3-8b-layer-quest", "quest", num_req=32, hq=32, hkv=8, head_dim=128, layers=1,
             steps=256, ctx=32768, top_k=64, relevant_pages=8, relevant_shift=3.0, seed=2),
    Workload(3, "ragged-continuous-batch-h2o", "h2o", num_req=128, hq=32, hkv=8, head_dim=128,
             layers=1, steps=128, ctx_log_range=(2048, 131072), retained_range=(1024, 4096),
             budget=4096, recent=512, hh_rate=0.01, hh_shift=4.0, seed=3),
    Workload(4, "llama3-8b-32-layer-h2o", "h2o", num_req=256, hq=32, hkv=8, head_dim=128, layers=32,
             steps=64, ctx=131072, initial_resident=4096, budget=4096, recent=512,
             hh_rate=0.01, hh_shift=4.0, seed=4),
]


# The decode workloads by name.
TINY_H2O, LAYER_H2O, LAYER_QUEST, RAGGED_H2O, MODEL_H2O = CONFIGS


# SnapKV prompt compaction after prefill (Appendix A.3, SnapKV; Appendix D uses
# a 32-token scoring window and pooling kernel 7): the prefilled prompt of
# every (request, KV head) is cut from 32768 slots to the 2048 that the H2O
# decode workload starts from, window 32 included.
SNAPKV = Workload(5, "llama3-8b-prompt-snapkv", "snapkv", num_req=64, hq=32, hkv=8, head_dim=128,
                  layers=1, steps=1, ctx=32768, budget=2048, obs_window=32, pool_kernel=7,
                  hh_rate=0.01, hh_shift=4.0, seed=5)


# OmniKV decode over a 32-layer 8B-shaped model (Appendix A.3, OmniKV; Appendix D:
# 2,048 selected tokens, Llama full-attention layers 0, 2, 7, 13, 16, 26): every
# request keeps its whole 32768-token history in every layer; observation layers
# attend densely and select b = 2048 slots, which the following sparse layers read.
OMNIKV = Workload(6, "llama3-8b-32-layer-omnikv", "omnikv", num_req=32, hq=32, hkv=8, head_dim=128,
                  layers=32, steps=32, ctx=32768, budget=2048, filter_layers=(0, 2, 7, 13, 16, 26),
                  hh_rate=0.01, hh_shift=4.0, seed=6)


# H2O chunk-wise prefill eviction (Appendix A.3, H2O; Appendix D, LongBench
# settings: 2,048-token budget, recent ratio 0.5, 8,192-token prefill chunks, a
# 128-query scoring window, FP32 scores): the fourth chunk of a 32768-token
# prompt has just been written behind the 2048 slots the earlier chunks left,
# 8 requests to a 65,536-token prefill step.  The call scores the 10240 slots
# with the chunk's last 128 queries of every head and cuts them back to 2048.
H2O_PREFILL = Workload(7, "llama3-8b-prefill-chunk-h2o", "h2o_prefill", num_req=8, hq=32, hkv=8, head_dim=128,
                       layers=1, steps=1, ctx=32768, initial_resident=2048 + 8192, budget=2048, recent=1024,
                       obs_window=128, chunk=8192, hh_rate=0.01, hh_shift=4.0, seed=7)


# Interval prefix-cache pruning (Section 3.2, "Sparsity-Based Prefix-Cache
# Pruning"; Appendix C.2): 8 idle agent chains of an 8B-shaped 32-layer model,
# each with its whole 32768-token history resident in every layer (slot s holds
# position s), prune a 4096-token tool-result interval [16384, 20480) to 20 % of
# its tokens (Section 4.3, "Quality of Prefix Pruning": 20 % of the targeted tool
# results' tokens retained; budget 819 per (layer, KV head) unit, the scoring
# policy's scores in the score field); the 12288 later slots close up behind it.
PRUNE = Workload(8, "llama3-8b-32-layer-prune-interval", "prune", num_req=8, hq=32, hkv=8, head_dim=128,
                 layers=32, steps=1, ctx=32768, budget=819, interval=(16384, 20480), seed=8)


def scaled(w: Workload, **changes) -> Workload:
    """A variant of a workload with some sizes changed (test cases)."""
    return replace(w, **changes)


def step_bounds(w: Workload, lengths, n: int):
    """Per-step upper bounds of any unit's resident slots after that step's
    append, as a scheduler knows them from the lengths at the start: H2O
    units grow by one per step up to the budget (then hold B + 1 after the
    append), Quest units grow by one per step.  ``lengths`` holds the initial
    resident slots of every unit (any integer sequence)."""
    L = max(int(x) for x in lengths)
    out = []
    for _ in range(int(n)):
        out.append(L + 1)
        L = min(L + 1, int(w.budget)) if w.method == "h2o" else L + 1
    return out
