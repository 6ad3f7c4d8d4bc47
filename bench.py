#!/usr/bin/env python3
"""Decode attention + eviction benchmark on one MI355X.

Default workload (the headline): the 32-layer Llama-3-8B-shaped H2O decode loop
(256 requests, Hq=32, Hkv=8, d=128, 4096 retained tokens per KV head and layer
of a 131072-token context, budget 4096 with a 512-token window; ~137 GB of KV
resident in HBM).  One timed step is one decode step of the whole batch
through all 32 layers: one se_decode_step_h2o call per layer (append,
attention, fused score update and one-slot eviction in one launch).  `value`
is requests x steps / wall time between device synchronisations; `roofline`
is the dominant kernel's algorithmic bytes per launch over its average launch
time (HIP events around the timed region, on the launch stream).  The
single-layer 8B-shaped workloads (H2O layer, Quest layer, ragged batch) run
after it with the same step counts and are reported under `other_configs`.

Protocol: the state is generated on the device (seeded); warm-up steps run on
a copy of a single-layer state (then dropped) or, for the 32-layer state, on
the state itself; the K timed steps then start with every input resident in
HBM, with the per-step length bound a scheduler knows (workloads.step_bounds).
`cpu_baseline` is the oracle on 64 units of the headline workload, timed on
the host before the GPU is touched and extrapolated to the whole batch.

Prints one JSON line.  `--config N` makes workload N (0..4) the headline;
`--workload omnikv` measures OmniKV decode over a 32-layer 8B-shaped model (32
requests, 32768-token histories, observation layers 0, 2, 7, 13, 16, 26
attend densely and select 2048 slots that the other layers read; one step is
one decode step through all 32 layers); `--workload snapkv` measures SnapKV
prompt compaction (se_snapkv_compact on the 8B-shaped prompt: 64 requests x 8
KV heads x 32768 slots, window 32, pooling width 7, budget 2048; one step is
one compaction of the whole batch from a fresh copy of the prompt);
`--workload h2o_prefill` measures H2O's chunk-wise prefill eviction
(se_h2o_prefill_chunk after the fourth 8192-token chunk of 32768-token
prompts, 8 requests x 8 KV heads, 2048 retained + 8192 chunk slots scored by
the chunk's last 128 queries of every head and cut back to 2048 with a
1024-token window; one step is one call from a fresh copy of that state);
`--workload prune` measures interval prefix-cache pruning (se_prune_interval
over 8 chains x 32 layers x 8 KV heads of 32768 resident slots: the interval
[16384, 20480) cut to its 819 best-scored slots per unit and the later slots
closed up; one step is one call from a fresh copy of the cache);
`--workload read_ceiling` measures a plain gather of random 8 KiB pages with
the decode stream's loads (se_probe_read_pages: the read rate the decode calls
are compared against); `--gpus N` with N > 1 is refused (single-GPU build).
"""

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "decode attn+eviction tokens/s/GPU; achieved HBM GB/s vs MI355X peak"
HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0
# Vector ALU: 256 compute units x 4 SIMDs x 16 lanes x 2.4 GHz = 39.3e12 lane-slots/s
# (one full-rate VALU operation per lane per slot; packed fp32, which would double
# fma and add, is not used by the library's kernels); v_exp_f32 takes two slots (measured on
# one MI355X: fma 3.99e13 lane-ops/s, exp2 alone 1.68e13/s, exp2 followed by two
# fma 1.06e13/s).
VALU_PEAK_TSLOTS = 256 * 4 * 16 * 2.4e9 / 1e12
VALU_SLOTS_PER_LOGIT = 2 * (2 + 1 + 1)
TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", "decode_step_h2o_llama3-8b-layer-h2o_traffic.txt")
SNAPKV_TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", "snapkv_compact_llama3-8b-prompt-snapkv_traffic.txt")
DECODE_SOURCES = ("decode_attend.hip", "evict_compact.hip", "evict_core.h", "quest_core.h", "se_common.h")
SNAPKV_SOURCES = ("snapkv.hip", "evict_compact.hip", "evict_core.h", "se_common.h")
PRUNE_TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", "prune_interval_llama3-8b-32-layer-prune-interval_traffic.txt")
PRUNE_SOURCES = ("prune.hip", "se_common.h")
OMNIKV_TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", "omnikv_step_llama3-8b-32-layer-omnikv_traffic.txt")
OMNIKV_SOURCES = ("decode_attend.hip", "omnikv.hip", "quest_core.h", "evict_core.h", "se_common.h")
PREFILL_TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", "h2o_prefill_chunk_llama3-8b-prefill-chunk-h2o_traffic.txt")


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None,
                    help="timed decode steps (default: 20 for the 32-layer workload, else the workload's)")
    ap.add_argument("--warmup", type=int, default=None, help="untimed steps (default 5; snapkv and prefill: 1)")
    ap.add_argument("--config", type=int, default=4, help="decode workload index 0..4 (default 4, the headline)")
    ap.add_argument("--only", action="store_true",
                    help="with --config 4: skip the single-layer workloads 1-3 reported under other_configs")
    ap.add_argument("--workload", choices=["decode", "snapkv", "omnikv", "h2o_prefill", "prune", "read_ceiling"],
                    default="decode",
                    help="decode (the --config workload), snapkv (prompt compaction), omnikv "
                         "(32-layer decode with OmniKV selection reuse), h2o_prefill (chunk-wise "
                         "prefill eviction), prune (interval prefix-cache pruning) or read_ceiling (the "
                         "plain read rate of the decode page gathers, se_probe_read_pages)")
    ap.add_argument("--cpu-baseline", choices=["auto", "skip"], default="auto")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run one plain 4 GiB device copy (counter calibration under rocprofv3)")
    return ap.parse_args()


# --------------------------------------------------------------------- CPU oracle baseline

def _oracle_unit_run(i):
    """One unit's trajectory through the oracle, in a forked worker that only
    touches NumPy arrays prepared by the parent."""
    from threadpoolctl import threadpool_limits
    from oracle import h2o, quest
    from oracle.state import new_unit
    job = _SHARED["jobs"][i]
    w = _SHARED["w"]
    with threadpool_limits(1):
        st = new_unit(job["K"], job["V"], job["pos"])
        if w.method == "quest":
            quest.attach_summaries(st)
        t0 = time.perf_counter()
        for t in range(len(job["p"])):
            if w.method == "h2o":
                h2o.decode_step(st, job["q"][t], job["k"][t], job["v"][t], job["p"][t], w.scale,
                                w.budget, w.recent)
            else:
                quest.decode_step(st, job["q"][t], job["k"][t], job["v"][t], job["p"][t], w.scale, w.top_k)
        return time.perf_counter() - t0


_SHARED = {}
CPU_SAMPLE_UNITS = 64


def cpu_baseline(w, K):
    """The oracle, untuned, on a bounded sample of the workload: 64 units of
    one layer (the first 64 // Hkv requests, every KV head, the workload's
    per-unit shapes and value recipe) for the same K decode steps, one unit per
    worker process, before the GPU is touched.  Units are independent, so the
    whole step extrapolates linearly: the mean CPU time per unit-step times the
    workload's units per layer and layers, spread over the worker processes,
    gives the oracle's full-batch step time; value = requests / that time."""
    import multiprocessing as mp
    import numpy as np
    import torch
    from workloads import build_state, build_steps, scaled, unit_slots
    sample_req = max(1, CPU_SAMPLE_UNITS // w.hkv)
    ws = scaled(w, num_req=sample_req, layers=1)
    host = build_state(ws, "cpu")
    steps = build_steps(ws, host, "cpu", steps=K)
    G = ws.q_per_kv

    def f64(t):
        return t.to(torch.float64).numpy()

    jobs = []
    for u in range(ws.units_per_layer):
        req, kvh = divmod(u, ws.hkv)
        Kt, Vt, pos, _ = unit_slots(host, u)
        jobs.append({"K": f64(Kt), "V": f64(Vt), "pos": pos.numpy().astype(np.int64),
                     "q": f64(steps.q[:, 0, req, kvh * G:(kvh + 1) * G]),
                     "k": f64(steps.k_new[:, 0, req, kvh]), "v": f64(steps.v_new[:, 0, req, kvh]),
                     "p": [int(x) for x in steps.new_pos[:, req]]})
    _SHARED["jobs"], _SHARED["w"] = jobs, ws
    workers = min(16, os.cpu_count() or 1, len(jobs))
    ctx = mp.get_context("fork")
    t0 = time.perf_counter()
    with ctx.Pool(workers) as pool:
        per_unit = pool.map(_oracle_unit_run, range(len(jobs)))
    wall = time.perf_counter() - t0
    unit_step_s = sum(per_unit) / (len(jobs) * K)
    step_s = unit_step_s * w.units_per_layer * w.layers / workers
    return {"value": round(w.num_req / step_s, 3), "unit": "tokens/s", "cores": workers, "kind": "oracle",
            "sample": (f"{len(jobs)} units (requests 0..{sample_req - 1}, all {ws.hkv} KV heads, one layer) of "
                       f"'{w.name}' for {K} decode steps each, NumPy float64, one unit per process; "
                       f"{1e3 * unit_step_s:.2f} ms per unit-step, extrapolated to {w.units_per_layer} units x "
                       f"{w.layers} layers on {workers} processes = {step_s:.3f} s per step of {w.num_req} requests"),
            "per_unit_step_ms": round(1e3 * unit_step_s, 3),
            "cpu_seconds": round(sum(per_unit), 2), "wall_seconds": round(wall, 2)}


# --------------------------------------------------------------------- algorithmic bytes

def h2o_step_bytes(L_pre, budget, G, D, moves):
    """Bytes one se_decode_step_h2o call must move for units holding L_pre
    slots before the step: every slot's K and V rows and its score read and
    written, plus its position where the unit evicts (L_pre + 1 > budget);
    per unit the G query rows (bf16), the G output rows (fp32) and the append
    (k, v read; k, v, position and score written); each moved slot's K, V,
    position and score read and written (``moves`` per unit)."""
    import numpy as np
    Lp = np.asarray(L_pre, dtype=np.int64) + 1
    ev = Lp > budget
    per_unit = G * D * 2 + G * D * 4 + 2 * D * 2 * 2 + 8
    move = 2 * (2 * D * 2 + 8)
    slots = int(Lp.sum()) * (2 * D * 2 + 8) + int(Lp[ev].sum()) * 4
    return slots + Lp.shape[0] * per_unit + int(np.asarray(moves).sum()) * move


def quest_step_bytes(L_pre, G, D, top_k):
    """Bytes one se_decode_step_quest call must move for units holding L_pre
    slots before the step: the min and max rows of every candidate page (the
    complete pages before the current one), the K and V rows of the top_k
    selected pages and of the current page's resident slots, the G query rows,
    the G output rows, the append (k, v read; k, v and position written; the
    current page's min and max read and written) and the selection written."""
    import numpy as np
    L = np.asarray(L_pre, dtype=np.int64)
    n_cand = L // 16
    visited = np.minimum(n_cand, top_k) * 16 + (L % 16 + 1)
    per_unit = G * D * 2 + G * D * 4 + 2 * D * 2 * 2 + 4 + 2 * (2 * D * 2) + top_k * 4
    return int(n_cand.sum()) * (2 * D * 2) + int(visited.sum()) * (2 * D * 2) + L.shape[0] * per_unit


def attend_kernel_name(units, n_visit, G, D, quest=False):
    """The decode_attend_kernel instantiation a launch of these sizes runs (the
    library's rule: 1024 threads when the units fit one work-group per compute
    unit, else 512; per-wavefront rows for the fused steady eviction when the
    largest wavefront slot's share of the pages fits them and every page's
    weights fit the LDS buffer; a Quest step's selection has its own)."""
    wide = units * -(-n_visit // 1024) <= 256
    nt = 1024 if wide else 512
    if quest:
        return f"decode_attend_kernel<{D},{G},{nt},false,true>"
    rows = (4 * 4 * 5 * 100 - 50) // (34 if wide else 58)
    wbytes = 4 if (nt == 512 and G <= 4) else 2  # fp32 or fp16 weights
    rows = min(rows, 1024, 9216 * 4 // wbytes // (16 * G))
    return f"decode_attend_kernel<{D},{G},{nt},{'true' if n_visit <= rows else 'false'},false>"


def snapkv_bytes(L, w, G, D, budget):
    """Bytes se_snapkv_compact must move for units of prompt length L > budget:
    the keys twice (the row normalisers need every key before any weight can
    be summed), the observation queries, u written and read back, each slot's
    position read and pooled score written; then the eviction's position and
    score reads and the movers' K, V, position and score read and written."""
    import numpy as np
    L = np.asarray(L, dtype=np.int64)
    L = L[L > budget]
    units = int(L.shape[0])
    score = int(L.sum()) * (2 * (D * 2) + 4 + 4 + 4 + 4) + units * (w * G * D * 2)
    moved = np.minimum(L - budget, budget)
    evict = int(L.sum()) * 8 + int(moved.sum()) * 2 * (2 * D * 2 + 8)
    return score + evict


def cpu_baseline_snapkv(w):
    """The oracle, untuned, on a bounded sample of the SnapKV workload: the
    first six requests (48 KV-head units of 32768 slots), one unit per worker
    process.  Runs before the GPU is touched."""
    import multiprocessing as mp
    import numpy as np
    import torch
    from workloads import build_observation, build_state, scaled, unit_slots
    sample_req = 6
    ws = scaled(w, num_req=sample_req)
    host = build_state(ws, "cpu")
    qobs = build_observation(ws, host, "cpu")
    G = ws.q_per_kv
    jobs = []
    for u in range(ws.units_per_layer):
        req, kvh = divmod(u, ws.hkv)
        Kt, Vt, pos, _ = unit_slots(host, u)
        jobs.append({"K": Kt.to(torch.float64).numpy(), "V": Vt.to(torch.float64).numpy(),
                     "pos": pos.numpy().astype(np.int64),
                     "Qo": qobs[req, :, kvh * G:(kvh + 1) * G].to(torch.float64).numpy()})
    _SHARED["jobs"], _SHARED["w"] = jobs, ws
    workers = min(16, os.cpu_count() or 1, len(jobs))
    ctx = mp.get_context("fork")
    t0 = time.perf_counter()
    with ctx.Pool(workers) as pool:
        per_unit = pool.map(_oracle_snapkv_run, range(len(jobs)))
    wall = time.perf_counter() - t0
    return {"value": round(sample_req * ws.ctx / wall, 1), "unit": "prompt tokens/s", "cores": workers,
            "kind": "oracle",
            "sample": (f"{sample_req} of {w.num_req} requests ({len(jobs)} KV-head units of {ws.ctx} slots) of "
                       f"'{w.name}', one compaction each, NumPy float64, one unit per process"),
            "cpu_seconds": round(sum(per_unit), 2), "wall_seconds": round(wall, 2)}


def _oracle_snapkv_run(i):
    from threadpoolctl import threadpool_limits
    from oracle import snapkv
    from oracle.state import new_unit
    job, w = _SHARED["jobs"][i], _SHARED["w"]
    with threadpool_limits(1):
        st = new_unit(job["K"], job["V"], job["pos"])
        t0 = time.perf_counter()
        snapkv.compact_prompt(st, job["Qo"], w.obs_window, w.pool_kernel, w.budget, w.scale)
        return time.perf_counter() - t0


def main_snapkv(args):
    """SnapKV prompt compaction: K compactions of the whole batch, each on a
    fresh copy of the prompt state made before its timed call."""
    from workloads import SNAPKV
    w = SNAPKV
    K = int(args.steps if args.steps is not None else 5)
    W = int(args.warmup if args.warmup is not None else 1)
    cpu = cpu_baseline_snapkv(w) if args.cpu_baseline == "auto" else None
    if cpu is not None:
        print(f"cpu baseline: {cpu['value']:.1f} prompt tokens/s on {cpu['cores']} processes", file=sys.stderr,
              flush=True)
    import numpy as np
    import torch
    import paper_2609_39068_amd as se
    from workloads import build_observation, build_state, clone_state

    assert torch.cuda.is_available(), "bench.py needs the GPU"
    dev = torch.device("cuda:0")
    state = build_state(w, dev)
    qobs = build_observation(w, state, dev)
    U, G, D = w.units_per_layer, w.q_per_kv, w.head_dim
    max_len = state.max_pages * 16
    ws = torch.empty(se.se_workspace_bytes(se.SE_OP_SNAPKV, U, max_len, state.max_pages, G, D),
                     dtype=torch.uint8, device=dev)
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    fcount = torch.zeros(U, dtype=torch.int32, device=dev)
    lengths0 = state.lengths.cpu().numpy()

    def call(st):
        view = se.KVView(st.kv_pool, st.pos_pool, st.score_pool, None, st.block_table, st.lengths,
                         num_kv_heads=w.hkv)
        se.se_snapkv_compact(view, G, qobs, w.obs_window, w.pool_kernel, w.scale, w.budget, max_len, 0,
                             None, 0, fcount, ws, err)

    for _ in range(W):
        c = clone_state(state)
        call(c)
        torch.cuda.synchronize()
        del c
    times, walls = [], []
    for _ in range(K):
        c = clone_state(state)
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        ev[0].record()
        call(c)
        ev[1].record()
        torch.cuda.synchronize()
        walls.append(time.perf_counter() - t0)
        times.append(ev[0].elapsed_time(ev[1]))
        assert int(c.lengths.max()) == w.budget
        del c
    errs = se.se_read_device_errors(err)
    if errs:
        raise RuntimeError(f"device error bits {errs:#x} during the timed run")
    ms = float(np.mean(times))
    elapsed = float(np.sum(walls))
    nbytes = snapkv_bytes(lengths0, w.obs_window, G, D, w.budget)
    achieved = nbytes / (ms * 1e-3) / 1e9
    result = {
        "metric": "SnapKV prompt compaction prompt-tokens/s/GPU; achieved HBM GB/s vs MI355X peak",
        "value": round(w.num_req * w.ctx * K / elapsed, 1),
        "unit": "prompt tokens/s",
        "n_gpus": 1, "steps": K, "warmup": W,
        "ms_per_step": round(1e3 * elapsed / K, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": w.name, "method": "snapkv", "batch": w.num_req, "hq": w.hq, "hkv": w.hkv,
                   "head_dim": D, "page_size": w.page_size, "prompt": w.ctx, "window": w.obs_window,
                   "pool_kernel": w.pool_kernel, "budget": w.budget, "accumulate": "f32",
                   "parallelism": "none (1 GPU)"},
        "roofline": {"bound": "hbm", "kernel": "se_snapkv_compact", "achieved": round(achieved, 1),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": read_traffic(SNAPKV_TRAFFIC_SUMMARY, SNAPKV_SOURCES),
                     "avg_launch_us": round(1e3 * ms, 3),
                     "algorithmic_bytes_per_launch": nbytes},
        "cpu_baseline": cpu,
    }
    if args.copy_calibration:
        n = 4 << 30
        a = torch.empty(n, dtype=torch.uint8, device=dev)
        b = torch.empty_like(a)
        b.copy_(a)
        torch.cuda.synchronize()
        result["copy_calibration_bytes"] = n
    print(json.dumps(result), flush=True)


def prefill_work(L, C, s, G, D, budget):
    """(bytes, flops) se_h2o_prefill_chunk must move and compute for units of L
    slots whose last C joined with this chunk, scored by s queries of each of
    the G heads.  Bytes: the keys twice (the row normalisers need every key
    before any weight can be summed), the queries, each slot's weight sum
    written and read back, the earlier slots' scores read and every score
    written; then the eviction's position and score reads and the movers' K, V,
    position and score read and written (units above the budget).  Flops: the
    s * G logit rows against every key once (2 * D per logit)."""
    import numpy as np
    L = np.asarray(L, dtype=np.int64)
    units = int(L.shape[0])
    score = int(L.sum()) * (2 * (D * 2) + 4 + 4 + 4) + int((L - C).clip(min=0).sum()) * 4 + units * (s * G * D * 2)
    over = L[L > budget]
    moved = np.minimum(over - budget, budget)
    evict = int(over.sum()) * 8 + int(moved.sum()) * 2 * (2 * D * 2 + 8)
    flops = int(L.sum()) * s * G * 2 * D
    return score + evict, flops


def cpu_baseline_h2o_prefill(w):
    """The oracle, untuned, on a bounded sample of the prefill workload: the
    first request (8 KV-head units), one unit per worker process, each
    taking the chunk's append, scoring and eviction.  Runs before the GPU is
    touched."""
    import multiprocessing as mp
    import numpy as np
    import torch
    from workloads import build_observation, build_state, scaled, unit_slots
    sample_req = 1
    ws = scaled(w, num_req=sample_req)
    host = build_state(ws, "cpu")
    qs = build_observation(ws, host, "cpu")
    G, C = ws.q_per_kv, ws.chunk
    jobs = []
    for u in range(ws.units_per_layer):
        req, kvh = divmod(u, ws.hkv)
        Kt, Vt, pos, sc = unit_slots(host, u)
        n0 = Kt.shape[0] - C
        f = lambda t: t.to(torch.float64).numpy()
        jobs.append({"K": f(Kt[:n0]), "V": f(Vt[:n0]), "pos": pos[:n0].numpy().astype(np.int64),
                     "u": sc[:n0].to(torch.float64).numpy(), "Kc": f(Kt[n0:]), "Vc": f(Vt[n0:]),
                     "pc": pos[n0:].numpy().astype(np.int64), "Qs": f(qs[req, :, kvh * G:(kvh + 1) * G])})
    _SHARED["jobs"], _SHARED["w"] = jobs, ws
    workers = min(16, os.cpu_count() or 1, len(jobs))
    ctx = mp.get_context("fork")
    t0 = time.perf_counter()
    with ctx.Pool(workers) as pool:
        per_unit = pool.map(_oracle_prefill_run, range(len(jobs)))
    wall = time.perf_counter() - t0
    return {"value": round(sample_req * C / wall, 1), "unit": "prompt tokens/s", "cores": workers,
            "kind": "oracle",
            "sample": (f"{sample_req} of {w.num_req} requests ({len(jobs)} KV-head units: {C}-token chunk behind "
                       f"{w.initial_resident - C} retained slots) of '{w.name}', one chunk each (append, "
                       f"scoring, eviction), NumPy float64, one unit per process"),
            "cpu_seconds": round(sum(per_unit), 2), "wall_seconds": round(wall, 2)}


def _oracle_prefill_run(i):
    from threadpoolctl import threadpool_limits
    from oracle import h2o
    from oracle.state import new_unit
    job, w = _SHARED["jobs"][i], _SHARED["w"]
    with threadpool_limits(1):
        st = new_unit(job["K"], job["V"], job["pos"], job["u"])
        t0 = time.perf_counter()
        h2o.prefill_chunk(st, job["Kc"], job["Vc"], job["pc"], job["Qs"], w.scale, w.budget, w.recent)
        return time.perf_counter() - t0


def main_h2o_prefill(args):
    """H2O chunk-wise prefill eviction: K calls over the whole batch, each on a
    fresh copy of the state (earlier retained slots + the chunk) made before
    its timed call."""
    from workloads import H2O_PREFILL
    w = H2O_PREFILL
    K = int(args.steps if args.steps is not None else 5)
    W = int(args.warmup if args.warmup is not None else 1)
    cpu = cpu_baseline_h2o_prefill(w) if args.cpu_baseline == "auto" else None
    if cpu is not None:
        print(f"cpu baseline: {cpu['value']:.1f} prompt tokens/s on {cpu['cores']} processes", file=sys.stderr,
              flush=True)
    import numpy as np
    import torch
    import paper_2609_39068_amd as se
    from workloads import build_observation, build_state, clone_state

    assert torch.cuda.is_available(), "bench.py needs the GPU"
    dev = torch.device("cuda:0")
    state = build_state(w, dev)
    qs = build_observation(w, state, dev)
    U, G, D, sw, C = w.units_per_layer, w.q_per_kv, w.head_dim, w.obs_window, w.chunk
    max_len = state.max_pages * 16
    ws = torch.empty(se.se_workspace_bytes(se.SE_OP_H2O_PREFILL, U, max_len, state.max_pages, G, D, sw),
                     dtype=torch.uint8, device=dev)
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    fcount = torch.zeros(U, dtype=torch.int32, device=dev)
    lengths0 = state.lengths.cpu().numpy()

    def call(st):
        view = se.KVView(st.kv_pool, st.pos_pool, st.score_pool, None, st.block_table, st.lengths,
                         num_kv_heads=w.hkv)
        se.se_h2o_prefill_chunk(view, G, qs, sw, C, w.scale, w.budget, w.recent, max_len, None, 0, fcount,
                                ws, err)

    for _ in range(W):
        c = clone_state(state)
        call(c)
        torch.cuda.synchronize()
        del c
    times, walls = [], []
    for _ in range(K):
        c = clone_state(state)
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        ev[0].record()
        call(c)
        ev[1].record()
        torch.cuda.synchronize()
        walls.append(time.perf_counter() - t0)
        times.append(ev[0].elapsed_time(ev[1]))
        assert int(c.lengths.max()) == w.budget
        del c
    errs = se.se_read_device_errors(err)
    if errs:
        raise RuntimeError(f"device error bits {errs:#x} during the timed run")
    ms = float(np.mean(times))
    elapsed = float(np.sum(walls))
    nbytes, flops = prefill_work(lengths0, C, sw, G, D, w.budget)
    achieved = nbytes / (ms * 1e-3) / 1e9
    # the binding resource: the vector ALU.  Every logit is exponentiated in both
    # passes (the row normaliser, then the weights), each time with one scale-and-
    # shift and one accumulation: 2 x (2 + 1 + 1) lane-slots, exp2 running at half
    # the full rate (at the peaks the ALU work takes 68 us, the HBM bytes 62 us and
    # the logit MFMAs 34 us)
    logits = flops // (2 * D)
    valu_slots = logits * VALU_SLOTS_PER_LOGIT
    alu_achieved = valu_slots / (ms * 1e-3) / 1e12
    result = {
        "metric": "H2O chunked-prefill eviction prompt-tokens/s/GPU; achieved vector-ALU rate vs MI355X peak",
        "value": round(w.num_req * C * K / elapsed, 1),
        "unit": "prompt tokens/s",
        "n_gpus": 1, "steps": K, "warmup": W,
        "ms_per_step": round(1e3 * elapsed / K, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": w.name, "method": "h2o_prefill", "batch": w.num_req, "hq": w.hq, "hkv": w.hkv,
                   "head_dim": D, "page_size": w.page_size, "prompt": w.ctx, "chunk": C,
                   "retained_before": w.initial_resident - C, "scoring_window": sw, "budget": w.budget,
                   "recent": w.recent, "accumulate": "f32", "parallelism": "none (1 GPU)"},
        "roofline": {"bound": "alu",
                     "kernel": "se_h2o_prefill_chunk (prefill_norm_kernel + prefill_score_kernel, then the eviction)",
                     "achieved": round(alu_achieved, 2), "peak": VALU_PEAK_TSLOTS,
                     "unit": "T VALU lane-slots/s", "frac": round(alu_achieved / VALU_PEAK_TSLOTS, 4),
                     "traffic": read_traffic(PREFILL_TRAFFIC_SUMMARY, SNAPKV_SOURCES),
                     "avg_launch_us": round(1e3 * ms, 3),
                     "algorithmic_valu_slots_per_launch": valu_slots,
                     "algorithmic_bytes_per_launch": nbytes,
                     "algorithmic_flops_per_launch": flops,
                     "hbm": {"achieved_GBps": round(achieved, 1), "frac": round(achieved / HBM_PEAK_GBS, 4)},
                     "mfma": {"achieved_TFLOPs": round(flops / (ms * 1e-3) / 1e12, 1),
                              "frac": round(flops / (ms * 1e-3) / 1e12 / MFMA_BF16_PEAK_TFLOPS, 4)}},
        "cpu_baseline": cpu,
    }
    if args.copy_calibration:
        n = 4 << 30
        a = torch.empty(n, dtype=torch.uint8, device=dev)
        b = torch.empty_like(a)
        b.copy_(a)
        torch.cuda.synchronize()
        result["copy_calibration_bytes"] = n
    print(json.dumps(result), flush=True)


def prune_bytes(L, n_t, moved, D):
    """Bytes se_prune_interval must move for units of L slots, n_t of them in
    the interval, `moved` of them changing slot: every position read once (to
    find the interval), the interval's scores read once (the selection), and
    each moved slot's key and value rows, position and score read and
    written."""
    import numpy as np
    L, n_t, moved = (np.asarray(x, dtype=np.int64) for x in (L, n_t, moved))
    return int(L.sum()) * 4 + int(n_t.sum()) * 4 + int(moved.sum()) * 2 * (4 * D + 8)


def cpu_baseline_prune(w):
    """The oracle, untuned, on a bounded sample of the pruning workload: the
    first layer's 64 units (8 chains x 8 KV heads), one unit per worker process,
    each taking the budget selection and the compaction.  Runs before the GPU is
    touched."""
    import multiprocessing as mp
    import numpy as np
    import torch
    from workloads import build_state, scaled, unit_slots
    ws = scaled(w, layers=1)
    host = build_state(ws, "cpu")
    jobs = []
    for u in range(ws.units_per_layer):
        Kt, Vt, pos, sc = unit_slots(host, u)
        jobs.append({"K": Kt.to(torch.float64).numpy(), "V": Vt.to(torch.float64).numpy(),
                     "pos": pos.numpy().astype(np.int64), "u": sc.to(torch.float64).numpy()})
    del host
    _SHARED["jobs"], _SHARED["w"] = jobs, ws
    workers = min(16, os.cpu_count() or 1, len(jobs))
    ctx = mp.get_context("fork")
    t0 = time.perf_counter()
    with ctx.Pool(workers) as pool:
        per_unit = pool.map(_oracle_prune_run, range(len(jobs)))
    wall = time.perf_counter() - t0
    lo, hi = w.interval
    share = len(jobs) / (w.layers * w.units_per_layer)      # of one call's units
    return {"value": round(share * w.num_req * (hi - lo) / wall, 1), "unit": "interval tokens/s",
            "cores": workers, "kind": "oracle",
            "sample": (f"layer 0 of {w.layers} ({len(jobs)} of {w.layers * w.units_per_layer} units, 32768 slots "
                       f"each) of '{w.name}', one pruning each (budget selection and compaction), NumPy float64, "
                       f"one unit per process; the rate is scaled by that share of a call"),
            "cpu_seconds": round(sum(per_unit), 2), "wall_seconds": round(wall, 2)}


def _oracle_prune_run(i):
    from threadpoolctl import threadpool_limits
    from oracle import prune
    from oracle.state import new_unit
    job, w = _SHARED["jobs"][i], _SHARED["w"]
    lo, hi = w.interval
    with threadpool_limits(1):
        st = new_unit(job["K"], job["V"], job["pos"], job["u"])
        t0 = time.perf_counter()
        prune.prune(st, lo, hi, prune.budget_selection(st, lo, hi, w.budget))
        return time.perf_counter() - t0


# Page gathers of the read-rate probe: (name, pages read, from a pool of, random order, work-groups).
# 526,336 pages = one 32-layer-workload layer-step (2048 units x 257 pages); 66,048 = one steady step of
# the 8B layer (512 units x 129 pages).
READ_CASES = [
    ("gather_4.3GB_random_of_17GB", 526336, 2097152, True, 2048),
    ("gather_0.54GB_random_of_17GB", 66048, 2097152, True, 512),
    ("stream_4.3GB", 526336, 2097152, False, 2048),
    ("gather_17GB_random", 2097152, 2097152, True, 8192),
]


def main_read_ceiling(args):
    """The plain read rate of the decode kernels' page gathers: se_probe_read_pages
    reads 8 KiB pages (a 16-slot page at d = 128) listed in a seeded random
    order from a 16 GiB pool with the decode stream's loads, K timed calls per
    case between HIP events.  `value` is the first case (one layer-step of the
    32-layer workload, 4.3 GB)."""
    import torch
    import paper_2609_39068_amd as se

    K = int(args.steps if args.steps is not None else 20)
    W = int(args.warmup if args.warmup is not None else 3)
    assert torch.cuda.is_available(), "bench.py needs the GPU"
    dev = torch.device("cuda:0")
    PB = 8192
    pool_pages = max(c[2] for c in READ_CASES)
    pool = torch.empty(pool_pages * PB, dtype=torch.uint8, device=dev)
    sink = torch.empty(max(c[4] for c in READ_CASES) * 512, dtype=torch.int32, device=dev)
    g = torch.Generator().manual_seed(7)
    cases = {}
    for name, n, of, rnd, grid in READ_CASES:
        pages = (torch.randperm(of, generator=g)[:n] if rnd else torch.arange(n)).to(torch.int32).to(dev)
        for _ in range(W):
            se.se_probe_read_pages(pool, pool_pages, pages, n, PB, grid, sink)
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        torch.cuda.synchronize()
        ev[0].record()
        for _ in range(K):
            se.se_probe_read_pages(pool, pool_pages, pages, n, PB, grid, sink)
        ev[1].record()
        torch.cuda.synchronize()
        us = 1e3 * ev[0].elapsed_time(ev[1]) / K
        cases[name] = {"pages": n, "bytes": n * PB, "pool_bytes": of * PB, "random": rnd, "work_groups": grid,
                       "us_per_call": round(us, 2), "GBps": round(n * PB / (us * 1e-6) / 1e9, 1)}
        print(f"{name}: {us:.1f} us, {cases[name]['GBps']} GB/s", file=sys.stderr, flush=True)
    head = cases[READ_CASES[0][0]]
    line = {"metric": "hbm_read_GBps", "value": head["GBps"], "unit": "GB/s", "n_gpus": 1, "steps": K, "warmup": W,
            "ms_per_step": round(head["us_per_call"] / 1e3, 4), "higher_is_better": True, "scaling": "weak",
            "vs_baseline": None, "dtype": "u8", "data": "synthetic",
            "config": {"workload": "read_ceiling", "page_bytes": PB, "parallelism": "none (1 GPU)"},
            "roofline": {"bound": "hbm", "kernel": "probe_read_kernel", "achieved": head["GBps"],
                         "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(head["GBps"] / HBM_PEAK_GBS, 4),
                         "traffic": None},
            "cases": cases}
    print(json.dumps(line))


def main_prune(args):
    """Interval prefix-cache pruning: K calls over every unit of every chain and
    layer, each on a fresh copy of the cache made before its timed call."""
    from workloads import PRUNE
    w = PRUNE
    K = int(args.steps if args.steps is not None else 5)
    W = int(args.warmup if args.warmup is not None else 1)
    cpu = cpu_baseline_prune(w) if args.cpu_baseline == "auto" else None
    if cpu is not None:
        print(f"cpu baseline: {cpu['value']:.1f} interval tokens/s on {cpu['cores']} processes", file=sys.stderr,
              flush=True)
    import numpy as np
    import torch
    import paper_2609_39068_amd as se
    from workloads import build_state, clone_state

    assert torch.cuda.is_available(), "bench.py needs the GPU"
    dev = torch.device("cuda:0")
    state = build_state(w, dev)
    U, D = w.layers * w.units_per_layer, w.head_dim
    lo, hi = w.interval
    max_len = state.max_pages * 16
    iv = torch.tensor([[lo, hi]] * U, dtype=torch.int32, device=dev)
    kb = torch.full((U,), w.budget, dtype=torch.int32, device=dev)
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    fcount = torch.zeros(U, dtype=torch.int32, device=dev)
    lengths0 = state.lengths.cpu().numpy()

    def call(st):
        view = se.KVView(st.kv_pool, st.pos_pool, st.score_pool, None, st.block_table, st.lengths,
                         num_kv_heads=w.hkv)
        se.se_prune_interval(view, iv, None, 0, kb, max_len, None, 0, fcount, err)

    moved = None
    for i in range(max(W, 1)):  # the first call (untimed) also gives the moved-slot count
        c = clone_state(state)
        call(c)
        torch.cuda.synchronize()
        if i == 0:
            # slot s held position s before the call: a slot whose position changed was written
            P = 16
            s = torch.arange(max_len, device=dev)
            pos = c.pos_pool[c.block_table.long()[:, s // P], s % P]
            moved = ((pos != s[None, :]) & (s[None, :] < c.lengths[:, None])).sum(dim=1).cpu().numpy()
        del c
    times, walls = [], []
    for _ in range(K):
        c = clone_state(state)
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        ev[0].record()
        call(c)
        ev[1].record()
        torch.cuda.synchronize()
        walls.append(time.perf_counter() - t0)
        times.append(ev[0].elapsed_time(ev[1]))
        assert int(c.lengths.max()) == w.ctx - (hi - lo) + w.budget
        del c
    errs = se.se_read_device_errors(err)
    if errs:
        raise RuntimeError(f"device error bits {errs:#x} during the timed run")
    ms = float(np.mean(times))
    elapsed = float(np.sum(walls))
    n_t = np.full(U, hi - lo)
    nbytes = prune_bytes(lengths0, n_t, moved, D)
    achieved = nbytes / (ms * 1e-3) / 1e9
    result = {
        "metric": "interval prefix-pruning interval-tokens/s/GPU; achieved HBM GB/s vs MI355X peak",
        "value": round(w.num_req * (hi - lo) * K / elapsed, 1),
        "unit": "interval tokens/s",
        "n_gpus": 1, "steps": K, "warmup": W,
        "ms_per_step": round(1e3 * elapsed / K, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": w.name, "method": "prune", "chains": w.num_req, "layers": w.layers, "hkv": w.hkv,
                   "head_dim": D, "page_size": w.page_size, "history": w.ctx, "interval": [lo, hi],
                   "budget": w.budget, "units": U, "parallelism": "none (1 GPU)"},
        "roofline": {"bound": "hbm", "kernel": "se_prune_interval", "achieved": round(achieved, 1),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": read_traffic(PRUNE_TRAFFIC_SUMMARY, PRUNE_SOURCES),
                     "avg_launch_us": round(1e3 * ms, 3),
                     "algorithmic_bytes_per_launch": nbytes, "moved_slots": int(moved.sum())},
        "cpu_baseline": cpu,
    }
    if args.copy_calibration:
        n = 4 << 30
        a = torch.empty(n, dtype=torch.uint8, device=dev)
        b = torch.empty_like(a)
        b.copy_(a)
        torch.cuda.synchronize()
        result["copy_calibration_bytes"] = n
    print(json.dumps(result), flush=True)


def omnikv_layer_bytes(L, G, D, b, observe):
    """Bytes one layer's OmniKV decode call(s) must move for units with L slots
    after the append.  Observation layer (se_decode_attend with logits, then
    se_omnikv_select): every slot's K and V rows and its G logits written, then
    read back, plus per request the max score written and read and the
    selection written.  Sparse layer (se_attend_slots): the b selected K and V
    rows.  Both: the G query rows, G output rows and lse, and the append (k, v
    read; k, v, position written)."""
    import numpy as np
    L = np.asarray(L, dtype=np.int64)
    units = int(L.shape[0])
    per_unit = G * D * 2 + G * D * 4 + G * 4 + 2 * D * 2 * 2 + 4
    if observe:
        return int(L.sum()) * (2 * D * 2 + 2 * G * 4) + units * per_unit
    return units * (int(b) * 2 * D * 2 + per_unit)


def cpu_baseline_omnikv(w, K):
    """The oracle, untuned, on a bounded sample of the OmniKV workload: two
    requests through one observation layer and one sparse layer (same shapes:
    32768-token histories, 8 KV heads, b = 2048) for K decode steps, one request
    per process; only the oracle's step calls are timed.  The per-token time of
    the 32-layer model is extrapolated as 6 observation + 26 sparse layers."""
    import multiprocessing as mp
    from workloads import build_state, build_steps, scaled
    sample_req = 2
    ws = scaled(w, num_req=sample_req, layers=2, filter_layers=(0,))
    host = build_state(ws, "cpu")
    steps = build_steps(ws, host, "cpu", steps=K)
    _SHARED["host"], _SHARED["steps"], _SHARED["w"], _SHARED["K"] = host, steps, ws, K
    ctx = mp.get_context("fork")
    t0 = time.perf_counter()
    with ctx.Pool(sample_req) as pool:
        per_req = pool.map(_oracle_omnikv_run, range(sample_req))
    wall = time.perf_counter() - t0
    n_obs = len(w.filter_layers)
    t_obs = sum(r[0] for r in per_req) / (sample_req * K)
    t_sparse = sum(r[1] for r in per_req) / (sample_req * K)
    per_token = n_obs * t_obs + (w.layers - n_obs) * t_sparse
    return {"value": round(sample_req / per_token, 4), "unit": "tokens/s", "cores": sample_req, "kind": "oracle",
            "sample": (f"{sample_req} of {w.num_req} requests of '{w.name}' through one observation and one sparse "
                       f"layer for {K} decode steps, NumPy float64, one request per process; the 32-layer token "
                       f"time is {n_obs} x observation ({t_obs:.3f} s) + {w.layers - n_obs} x sparse "
                       f"({t_sparse:.4f} s), and value = processes / that time"),
            "cpu_seconds": round(sum(r[0] + r[1] for r in per_req), 2), "wall_seconds": round(wall, 2)}


def _oracle_omnikv_run(r):
    import numpy as np
    import torch
    from threadpoolctl import threadpool_limits
    from oracle import omnikv
    from oracle.state import new_unit
    from workloads import unit_slots
    host, steps, w, K = _SHARED["host"], _SHARED["steps"], _SHARED["w"], _SHARED["K"]
    U = w.units_per_layer

    def f64(t):
        return t.to(torch.float64).numpy()

    spent = [0.0, 0.0]   # observation, sparse
    J = {}
    with threadpool_limits(1):
        for layer in range(w.layers):
            units = []
            for h in range(w.hkv):
                Kt, Vt, pos, _ = unit_slots(host, layer * U + r * w.hkv + h)
                units.append(new_unit(f64(Kt), f64(Vt), pos.numpy().astype(np.int64)))
            for t in range(K):
                q, kn, vn = f64(steps.q[t, layer, r]), f64(steps.k_new[t, layer, r]), f64(steps.v_new[t, layer, r])
                p = int(steps.new_pos[t, r])
                t0 = time.perf_counter()
                if layer in w.filter_layers:
                    J[t] = omnikv.filter_step(units, q, kn, vn, p, w.scale, w.budget)["J"]
                    spent[0] += time.perf_counter() - t0
                else:
                    omnikv.sparse_step(units, q, kn, vn, p, w.scale, J[t])
                    spent[1] += time.perf_counter() - t0
    return spent


def main_omnikv(args):
    """K decode steps of the OmniKV workload through all layers; the state keeps
    growing (one appended token per layer and step), so warm-up steps run on the
    state itself before the timed ones."""
    from workloads import OMNIKV
    w = OMNIKV
    K = int(args.steps if args.steps is not None else 8)
    W = int(args.warmup if args.warmup is not None else 2)
    if K + W > w.steps:
        raise SystemExit(f"bench.py: --steps + --warmup must be at most {w.steps} (the slots reserved per unit)")
    cpu = cpu_baseline_omnikv(w, 1) if args.cpu_baseline == "auto" else None
    if cpu is not None:
        print(f"cpu baseline: {cpu['value']:.3f} tokens/s", file=sys.stderr, flush=True)
    import numpy as np
    import torch
    import paper_2609_39068_amd as se
    from workloads import build_state, build_steps

    assert torch.cuda.is_available(), "bench.py needs the GPU"
    dev = torch.device("cuda:0")
    t_gen = time.perf_counter()
    state = build_state(w, dev)
    steps = build_steps(w, state, dev, steps=W + K)
    torch.cuda.synchronize()
    print(f"generated '{w.name}' in {time.perf_counter() - t_gen:.1f}s", file=sys.stderr, flush=True)
    U, G, D, b = w.units_per_layer, w.q_per_kv, w.head_dim, w.budget
    max_len = state.max_pages * 16
    views = [se.KVView(state.kv_pool, state.pos_pool, None, None, state.block_table[state.layer_rows(l)],
                       state.lengths[state.layer_rows(l)], num_kv_heads=w.hkv) for l in range(w.layers)]
    out = torch.empty((w.num_req, w.hq, D), dtype=torch.float32, device=dev)
    lse = torch.empty((w.num_req, w.hq), dtype=torch.float32, device=dev)
    dec = se.OmniKVDecoder(G, w.scale, b, w.filter_layers, U, w.hkv, max_len, state.max_pages, D, dev)
    err = dec.dev_err
    observe = set(w.filter_layers)

    def run(t0, t1, lengths, layer_events=None, span=None):
        for t in range(t0, t1):
            ml = int(lengths) + (t - t0) + 1
            if span is not None and t == t0:
                span[0].record()
            for l in range(w.layers):
                dec.layer(l, views[l], steps.q[t, l], steps.k_new[t, l], steps.v_new[t, l], steps.new_pos[t], out,
                          lse, ml)
                if layer_events is not None and t == t0:
                    layer_events[l].record()
            if span is not None:
                if t == t0:
                    span[1].record()
                if t == t1 - 1:
                    span[2].record()

    L0 = int(state.lengths.max())
    run(0, W, L0)
    torch.cuda.synchronize()
    lengths0 = state.lengths.cpu().numpy().astype(np.int64).reshape(w.layers, U)
    span = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    lev = [torch.cuda.Event(enable_timing=True) for _ in range(w.layers)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    run(W, W + K, int(lengths0.max()), lev, span)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    errs = se.se_read_device_errors(err)
    if errs:
        raise RuntimeError(f"device error bits {errs:#x} during the timed run")
    region_ms = span[0].elapsed_time(span[2])
    # per-layer times of the first timed step (events after each layer)
    obs_ms = sparse_ms = 0.0
    for l in range(w.layers):
        ms = span[0].elapsed_time(lev[0]) if l == 0 else lev[l - 1].elapsed_time(lev[l])
        if l in observe:
            obs_ms += ms
        else:
            sparse_ms += ms
    total = obs_bytes = sparse_bytes = 0
    for t in range(K):
        for l in range(w.layers):
            Lp = lengths0[l] + t + 1
            nb = omnikv_layer_bytes(Lp, G, D, b, l in observe)
            total += nb
            if t == 0:
                if l in observe:
                    obs_bytes += nb
                else:
                    sparse_bytes += nb
    achieved = total / (region_ms * 1e-3) / 1e9
    result = {
        "metric": "OmniKV decode tokens/s/GPU (32 layers); achieved HBM GB/s vs MI355X peak",
        "value": round(w.num_req * K / elapsed, 1),
        "unit": "tokens/s",
        "n_gpus": 1, "steps": K, "warmup": W,
        "ms_per_step": round(1e3 * elapsed / K, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": w.name, "method": "omnikv", "batch": w.num_req, "hq": w.hq, "hkv": w.hkv,
                   "head_dim": D, "page_size": w.page_size, "layers": w.layers, "context": w.ctx,
                   "selected": b, "observation_layers": list(w.filter_layers), "accumulate": "f32",
                   "parallelism": "none (1 GPU)"},
        "roofline": {"bound": "hbm", "kernel": "OmniKV decode step (se_decode_attend + se_omnikv_select on "
                                               "observation layers, se_attend_slots on the others)",
                     "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": read_traffic(OMNIKV_TRAFFIC_SUMMARY, OMNIKV_SOURCES),
                     "avg_launch_us": round(1e3 * region_ms / K, 3),
                     "algorithmic_bytes_per_launch": round(total / K)},
        "phases": {"observation_layers_ms": round(obs_ms, 3),
                   "observation_GBps": round(obs_bytes / (obs_ms * 1e-3) / 1e9, 1),
                   "sparse_layers_ms": round(sparse_ms, 3),
                   "sparse_GBps": round(sparse_bytes / (sparse_ms * 1e-3) / 1e9, 1)},
        "cpu_baseline": cpu,
    }
    if args.copy_calibration:
        n = 4 << 30
        a = torch.empty(n, dtype=torch.uint8, device=dev)
        bb = torch.empty_like(a)
        bb.copy_(a)
        torch.cuda.synchronize()
        result["copy_calibration_bytes"] = n
    print(json.dumps(result), flush=True)


def source_hash(files=DECODE_SOURCES):
    h = hashlib.sha256()
    for f in files:
        h.update(open(os.path.join(ROOT, "paper_2609_39068_amd", "csrc", f), "rb").read())
    return h.hexdigest()[:16]


def read_summary(path, files=DECODE_SOURCES):
    """The numeric fields of a committed rocprofv3 counter summary, or None when
    it is missing or the kernels have changed since it was taken."""
    if not os.path.exists(path):
        return None
    vals = {}
    for line in open(path):
        if "=" in line and not line.lstrip().startswith("#"):
            k, v = line.split("=", 1)
            vals[k.strip()] = v.strip()
    if vals.get("source_hash") != source_hash(files):
        return None
    out = {}
    for k, v in vals.items():
        try:
            out[k] = float(v)
        except ValueError:
            pass
    return out


def read_traffic(path=TRAFFIC_SUMMARY, files=DECODE_SOURCES):
    """HBM bytes per call from a committed counter summary (or None)."""
    vals = read_summary(path, files)
    return None if vals is None else vals.get("hbm_bytes_per_launch")


def decode_traffic_path(w):
    return os.path.join(ROOT, "profiles", f"decode_step_{w.method}_{w.name}_traffic.txt")


def split_count(units, n_visit):
    """Work-groups per unit of a decode launch (the library's split rule)."""
    wide = units * -(-n_visit // 1024) <= 256
    resident = 256 if wide else 512
    splits = min(-(-resident // units), -(-n_visit // 16))
    splits = max(splits, 1, -(-n_visit // 1024))
    pps = -(-n_visit // splits)
    return -(-n_visit // pps)


# --------------------------------------------------------------------- GPU run

def slot_positions(st, n):
    """int32 [units, n]: the positions of every unit's slots [0, n)."""
    import torch
    s = torch.arange(n, device=st.block_table.device)
    page = st.block_table[:, :(n + 15) // 16].to(torch.int64)[:, s // 16]
    return st.pos_pool[page, (s % 16)[None, :].expand_as(page)]


def run_decode(w, K, W, se, dev):
    """K timed decode steps of workload w (every layer, one call per layer and
    step) after W warm-up steps; returns the measurement (no tensors)."""
    import numpy as np
    import torch
    from workloads import build_state, build_steps, clone_state, step_bounds

    t_gen = time.perf_counter()
    state = build_state(w, dev)
    keep_going = w.layers > 1          # too large to copy: warm up on the state itself
    n_inputs = K + W if keep_going else max(K, W, 1)
    steps = build_steps(w, state, dev, steps=n_inputs)
    torch.cuda.synchronize()
    print(f"generated '{w.name}' in {time.perf_counter() - t_gen:.1f}s", file=sys.stderr, flush=True)

    U, G, D = w.units_per_layer, w.q_per_kv, w.head_dim
    max_len = state.max_pages * 16
    out = torch.empty((w.num_req, w.hq, D), dtype=torch.float32, device=dev)

    def make(st):
        views = [se.KVView(st.kv_pool, st.pos_pool, st.score_pool, st.meta_pool,
                           st.block_table[st.layer_rows(l)], st.lengths[st.layer_rows(l)],
                           num_kv_heads=w.hkv) for l in range(w.layers)]
        if w.method == "h2o":
            ws = se.H2ODecoder.workspace(views[0], G, max_len, dev)
            err = torch.zeros(1, dtype=torch.int32, device=dev)
            return [se.H2ODecoder(v, G, w.scale, w.budget, w.recent, max_len, dev, ws=ws, dev_err=err)
                    for v in views]
        decs = [se.QuestDecoder(v, G, w.scale, w.top_k, max_len, dev) for v in views]
        for d in decs:
            d.summarize()
        return decs

    def run(decs, t0, t1, bounds, span=None):
        """One call per layer and step (se_decode_step_h2o / se_decode_step_quest)
        with the step's length bound.  span: events before the first step, after
        it and after the last (an event costs a few microseconds of GPU time, so
        calls are not bracketed one by one)."""
        for t in range(t0, t1):
            ml = bounds[t - t0]
            if span is not None and t == t0:
                span[0].record()
            for l, d in enumerate(decs):
                d.step(steps.q[t, l], steps.k_new[t, l], steps.v_new[t, l], steps.new_pos[t], out, max_len=ml)
            if span is not None:
                if t == t0:
                    span[1].record()
                if t == t1 - 1:
                    span[2].record()

    host_len = state.lengths.cpu().numpy().astype(np.int64)
    # the first step is not the steady one when a unit holds more than B + 1
    # slots after its append: count the slots it moves (the compaction's
    # movers) on the warm-up copy, which takes the same step on the same inputs
    first_general = w.method == "h2o" and int(host_len.max()) + 1 > w.budget + 1
    moves1 = None
    t_base = 0
    if keep_going:
        if first_general:
            raise SystemExit("bench.py: a multi-layer workload must start in the steady state")
        decs = make(state)
        if W > 0:
            run(decs, 0, W, step_bounds(w, host_len, W))
            t_base = W
    else:
        scratch = clone_state(state)
        sdecs = make(scratch)
        bw = step_bounds(w, host_len, max(W, 1))
        if first_general:
            before = slot_positions(scratch, w.budget)
            run(sdecs, 0, 1, bw[:1])
            after = slot_positions(scratch, w.budget)
            moves1 = (before != after).sum(dim=1).cpu().numpy() * (host_len + 1 > w.budget)
            run(sdecs, 1, W, bw[1:])
        else:
            run(sdecs, 0, W, bw)
        torch.cuda.synchronize()
        del scratch, sdecs
        torch.cuda.empty_cache()
        decs = make(state)
    torch.cuda.synchronize()
    lengths0 = state.lengths.cpu().numpy().astype(np.int64).reshape(w.layers, U)
    bounds = step_bounds(w, lengths0.reshape(-1), K)

    span = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    run(decs, t_base, t_base + K, bounds, span)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    errs = se.se_read_device_errors(decs[0].dev_err)
    if errs:
        raise RuntimeError(f"device error bits {errs:#x} during the timed run")
    step1_ms = span[0].elapsed_time(span[1])
    region_ms = span[0].elapsed_time(span[2])

    # algorithmic bytes per step (lengths follow the method's rule on the host)
    L = lengths0.copy()
    step_bytes = []
    for t in range(K):
        b = 0
        for l in range(w.layers):
            if w.method == "h2o":
                # a steady step moves one slot per evicting unit (the newest slot,
                # always in the window, fills the victim's)
                mv = moves1 if (t == 0 and moves1 is not None) else (L[l] + 1 > w.budget).astype(np.int64)
                b += h2o_step_bytes(L[l], w.budget, G, D, mv)
                L[l] = np.minimum(L[l] + 1, w.budget)
            else:
                b += quest_step_bytes(L[l], G, D, w.top_k)
                L[l] = L[l] + 1
        step_bytes.append(b)

    def n_visit_of(ml):
        return w.top_k + 1 if w.method == "quest" else -(-min(ml, max_len) // 16)

    def kernels(ml):
        nv = n_visit_of(ml)
        name = attend_kernel_name(U, nv, G, D, quest=w.method == "quest")
        if w.method == "quest":
            return name + " (page bounds, top-k and attention)"
        ns = split_count(U, nv)
        if ns > 1:
            return f"{name} x {ns} work-groups per unit + decode_combine_kernel + evict_compact_kernel"
        return name + " (score update and eviction in the epilogue)"

    calls = w.layers
    traffic = read_summary(decode_traffic_path(w))
    phases = {}
    if moves1 is not None and K > 1:
        steady_ms = region_ms - step1_ms
        sb = sum(step_bytes[1:])
        phases["step1"] = {"kernels": kernels(bounds[0]), "ms": round(step1_ms, 4),
                           "algorithmic_bytes_per_launch": step_bytes[0] // calls,
                           "moved_slots": int(moves1.sum()),
                           "GBps": round(step_bytes[0] / (step1_ms * 1e-3) / 1e9, 1),
                           "traffic": None if traffic is None else traffic.get("hbm_bytes_step1")}
        phases["steady"] = {"kernels": kernels(bounds[1]), "ms_per_step": round(steady_ms / (K - 1), 4),
                            "algorithmic_bytes_per_launch": round(sb / ((K - 1) * calls)),
                            "GBps": round(sb / (steady_ms * 1e-3) / 1e9, 1),
                            "traffic": None if traffic is None else traffic.get("hbm_bytes_steady")}
        dom_ms, dom_bytes, dom_launches, dom_ml = steady_ms, sb, (K - 1) * calls, bounds[1]
    else:
        dom_ms, dom_bytes, dom_launches, dom_ml = region_ms, sum(step_bytes), K * calls, bounds[0]
    achieved = dom_bytes / (dom_ms * 1e-3) / 1e9
    roof = {"bound": "hbm", "kernel": attend_kernel_name(U, n_visit_of(dom_ml), G, D, quest=w.method == "quest"),
            "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": None if traffic is None else traffic.get("hbm_bytes_steady"),
            "avg_launch_us": round(1e3 * dom_ms / dom_launches, 3),
            "algorithmic_bytes_per_launch": round(dom_bytes / dom_launches),
            "launches": dom_launches,
            "window": "steady steps 2..K" if moves1 is not None and K > 1 else "all timed steps"}
    return {"w": w, "value": w.num_req * K / elapsed, "ms_per_step": 1e3 * elapsed / K, "region_ms": region_ms,
            "roofline": roof, "phases": phases, "step_GBps": round(sum(step_bytes) / elapsed / 1e9, 1)}


def config_fields(w):
    return {"workload": w.name, "method": w.method, "batch": w.num_req, "hq": w.hq, "hkv": w.hkv,
            "head_dim": w.head_dim, "page_size": w.page_size, "layers": w.layers,
            "context": w.ctx if w.ctx is not None else list(w.ctx_log_range),
            "resident": w.initial_resident if w.initial_resident is not None else w.retained_range,
            "budget": w.budget, "recent": w.recent, "top_k": w.top_k, "accumulate": "f32",
            "parallelism": "none (1 GPU)"}


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: every unit (request, KV head) is independent, "
              "so N GPUs would each run this same benchmark on their share of the requests. "
              "Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)
    if args.workload == "snapkv":
        main_snapkv(args)
        return
    if args.workload == "omnikv":
        main_omnikv(args)
        return
    if args.workload == "h2o_prefill":
        main_h2o_prefill(args)
        return
    if args.workload == "prune":
        main_prune(args)
        return
    if args.workload == "read_ceiling":
        main_read_ceiling(args)
        return
    from workloads import CONFIGS
    w = CONFIGS[args.config]
    K = int(args.steps if args.steps is not None else (20 if w.layers > 1 else w.steps))
    W = int(args.warmup if args.warmup is not None else 5)
    if w.layers > 1 and K + W > w.steps:
        raise SystemExit(f"bench.py: --steps + --warmup must be at most {w.steps} for '{w.name}'")

    cpu = None
    if args.cpu_baseline == "auto":
        cpu = cpu_baseline(w, K)
        print(f"cpu baseline: {cpu['value']:.3f} tokens/s on {cpu['cores']} processes", file=sys.stderr,
              flush=True)

    import torch
    import paper_2609_39068_amd as se

    assert torch.cuda.is_available(), "bench.py needs the GPU"
    dev = torch.device("cuda:0")
    r = run_decode(w, K, W, se, dev)
    torch.cuda.empty_cache()
    result = {
        "metric": METRIC,
        "value": round(r["value"], 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": round(r["ms_per_step"], 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": config_fields(w),
        "roofline": r["roofline"],
        "step_GBps": r["step_GBps"],
        "cpu_baseline": cpu,
    }
    if r["phases"]:
        result["phases"] = r["phases"]
    if args.config == 4 and not args.only:
        # the single-layer 8B-shaped workloads, same step counts
        others = {}
        for idx in (1, 2, 3):
            wo = CONFIGS[idx]
            ro = run_decode(wo, K, W, se, dev)
            torch.cuda.empty_cache()
            e = {"config": config_fields(wo), "value": round(ro["value"], 1), "unit": "per-layer tokens/s",
                 "ms_per_step": round(ro["ms_per_step"], 4), "roofline": ro["roofline"]}
            if ro["phases"]:
                e["phases"] = ro["phases"]
            others[wo.name] = e
            print(f"{wo.name}: {ro['value']:.0f} per-layer tokens/s, {ro['roofline']['frac']:.3f} of HBM peak",
                  file=sys.stderr, flush=True)
        result["other_configs"] = others
    if args.copy_calibration:
        n = 4 << 30
        a = torch.empty(n, dtype=torch.uint8, device=dev)
        b = torch.empty_like(a)
        b.copy_(a)
        torch.cuda.synchronize()
        result["copy_calibration_bytes"] = n
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
