"""The five workloads at their full sizes, in the launch configuration the
benchmark times, checked against the oracle on sampled units.

Inputs are generated on the device by the seeded generators; the sampled
units' initial state and per-step inputs are copied back before any library
call runs, and the oracle steps each sampled unit on its own.
"""
import numpy as np
import pytest
import torch

from oracle import h2o, quest
from tests.oracle_bridge import (OUT_ATOL, QUEST_RTOL, assert_scores_close, f64, gpu_unit,
                                 h2o_near_tie, oracle_unit, quest_near_tie)
from workloads import LAYER_H2O, LAYER_QUEST, MODEL_H2O, RAGGED_H2O, build_state, build_steps

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


@pytest.fixture(scope="module")
def se():
    import paper_2609_39068_amd as m
    assert torch.cuda.is_available()
    return m


def _layer_view(se, gs, layer):
    rows = gs.layer_rows(layer)
    return se.KVView(gs.kv_pool, gs.pos_pool, gs.score_pool, gs.meta_pool, gs.block_table[rows],
                     gs.lengths[rows], num_kv_heads=gs.w.hkv)


def _sample(w, n, seed):
    g = torch.Generator().manual_seed(seed)
    picks = set()
    while len(picks) < n:
        layer = int(torch.randint(0, w.layers, (1,), generator=g))
        unit = int(torch.randint(0, w.units_per_layer, (1,), generator=g))
        picks.add((layer, unit))
    return sorted(picks)


def _run_h2o_sampled(se, w, n_steps, n_sample):
    print(f"generating {w.name}", flush=True)
    gs = build_state(w, DEV)
    steps = build_steps(w, gs, DEV, steps=n_steps)
    sample = _sample(w, n_sample, seed=w.seed + 99)
    U, G = w.units_per_layer, w.q_per_kv
    ost = {(l, u): oracle_unit(gs, l * U + u) for l, u in sample}
    max_len = gs.max_pages * 16
    views = [_layer_view(se, gs, l) for l in range(w.layers)]
    ws = se.H2ODecoder.workspace(views[0], G, max_len, DEV)
    decs = [se.H2ODecoder(v, G, w.scale, w.budget, w.recent, max_len, DEV, ws=ws) for v in views]
    out = torch.empty((w.num_req, w.hq, w.head_dim), dtype=torch.float32, device=DEV)
    checked, diverged = 0, set()
    for t in range(n_steps):
        print(f"step {t}", flush=True)
        for l in range(w.layers):
            decs[l].attend(steps.q[t, l], steps.k_new[t, l], steps.v_new[t, l], steps.new_pos[t], out)
            torch.cuda.synchronize()
            layer_units = [u for (ll, u) in sample if ll == l and (ll, u) not in diverged]
            pre = {u: gpu_unit(gs, l * U + u) for u in layer_units}
            o_g = out.cpu().double().numpy()
            decs[l].evict()
            torch.cuda.synchronize()
            assert se.se_read_device_errors(decs[l].dev_err) == 0
            for u in layer_units:
                req, kvh = divmod(u, w.hkv)
                rows = slice(kvh * G, (kvh + 1) * G)
                st = ost[(l, u)]
                res = h2o.decode_step(st, f64(steps.q[t, l, req, rows]), f64(steps.k_new[t, l, req, kvh]),
                                      f64(steps.v_new[t, l, req, kvh]), int(steps.new_pos[t, req]),
                                      w.scale, w.budget, w.recent)
                assert np.abs(o_g[req, rows] - res["o"]).max() <= OUT_ATOL, (t, l, u)
                np.testing.assert_array_equal(pre[u]["pos"], res["pos_after_append"])
                assert_scores_close(pre[u]["u"], res["u_after_accumulate"], f"{t} {l} {u}")
                after = gpu_unit(gs, l * U + u)
                kg, ko = set(after["pos"].tolist()), set(st.pos.tolist())
                if kg != ko:
                    ou = dict(zip(res["pos_after_append"].tolist(), res["u_after_accumulate"].tolist()))
                    assert h2o_near_tie(ou, kg, ko), f"step {t} layer {l} unit {u}: retained sets differ"
                    diverged.add((l, u))
                    continue
                np.testing.assert_array_equal(after["pos"], st.pos)
                np.testing.assert_array_equal(after["K"], st.K)
                np.testing.assert_array_equal(after["V"], st.V)
                checked += 1
    return checked, diverged


def test_8b_layer_h2o_full_size(se):
    # 64 requests x 8 KV heads, 32768-token contexts: step 1 evicts 32769 -> 2048
    # (radix path), step 2 is the steady one-slot eviction.
    w = LAYER_H2O
    checked, diverged = _run_h2o_sampled(se, w, 2, 8)
    assert len(diverged) <= 2 and checked >= 12


def test_ragged_batch_h2o_full_size(se):
    # 128 requests, ragged per-head lengths 1024..4096, budget 4096.
    w = RAGGED_H2O
    checked, diverged = _run_h2o_sampled(se, w, 2, 12)
    assert len(diverged) <= 2 and checked >= 20


def test_32_layer_h2o_full_size(se):
    # 32 layers x 256 requests x 8 KV heads at 4096 retained tokens (~137 GB of KV).
    w = MODEL_H2O
    checked, diverged = _run_h2o_sampled(se, w, 2, 12)
    assert len(diverged) <= 2 and checked >= 20


def test_8b_layer_quest_full_size(se):
    # Quest over 2048 pages per KV head, top-64, 32 requests.
    w = LAYER_QUEST
    print(f"generating {w.name}", flush=True)
    gs = build_state(w, DEV)
    steps = build_steps(w, gs, DEV, steps=2)
    U, G = w.units_per_layer, w.q_per_kv
    sample = [u for (_, u) in _sample(w, 8, seed=w.seed + 99)]
    ost = {u: oracle_unit(gs, u) for u in sample}
    for st in ost.values():
        quest.attach_summaries(st)
    dec = se.QuestDecoder(_layer_view(se, gs, 0), G, w.scale, w.top_k, gs.max_pages * 16, DEV)
    dec.summarize()
    scores = torch.empty((U, gs.max_pages), dtype=torch.float32, device=DEV)
    out = torch.empty((w.num_req, w.hq, w.head_dim), dtype=torch.float32, device=DEV)
    same = 0
    for t in range(2):
        print(f"step {t}", flush=True)
        dec.select(steps.q[t, 0], scores)
        dec.attend(steps.q[t, 0], steps.k_new[t, 0], steps.v_new[t, 0], steps.new_pos[t], out)
        torch.cuda.synchronize()
        assert se.se_read_device_errors(dec.dev_err) == 0
        o_g = out.cpu().double().numpy()
        for u in sample:
            req, kvh = divmod(u, w.hkv)
            rows = slice(kvh * G, (kvh + 1) * G)
            res = quest.decode_step(ost[u], f64(steps.q[t, 0, req, rows]), f64(steps.k_new[t, 0, req, kvh]),
                                    f64(steps.v_new[t, 0, req, kvh]), int(steps.new_pos[t, req]),
                                    w.scale, w.top_k)
            n = res["n_candidates"]
            sc = scores[u, :n].cpu().double().numpy()
            assert (np.abs(sc - res["scores"]) / np.maximum(1, np.abs(res["scores"]))).max() <= QUEST_RTOL
            got = dec.sel[u].cpu().numpy()
            if got.tolist() != res["selected"].tolist():
                assert quest_near_tie(res["scores"], got, res["selected"])
                continue
            same += 1
            assert np.abs(o_g[req, rows] - res["o"]).max() <= OUT_ATOL
    assert same >= 12
