"""SnapKV prompt compaction on the GPU against the oracle: se_snapkv_compact
(observation-window scores, max pooling, retention with the window, H2O's
compaction), in score-only mode and in full.

Every input comes from the seeded generators in workloads/; the oracle reads
them before any library call touches them.
"""
import numpy as np
import pytest
import torch

from oracle import snapkv
from tests.oracle_bridge import assert_scores_close, f64, gpu_unit, h2o_near_tie, oracle_unit
from workloads import (SNAPKV, build_observation, build_state, clone_state, isolated_units,
                       observation_queries, scaled, to_device)

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


@pytest.fixture(scope="module")
def se():
    import paper_2609_39068_amd as m
    assert torch.cuda.is_available()
    return m


def _view(se, st, hkv):
    return se.KVView(st.kv_pool, st.pos_pool, st.score_pool, None, st.block_table, st.lengths,
                     num_kv_heads=hkv)


def _call(se, gs, hkv, G, qobs, window, kappa, scale, budget, flags=0):
    U = gs.lengths.numel()
    max_len = gs.max_pages * 16
    ws = torch.empty(se.se_workspace_bytes(se.SE_OP_SNAPKV, U, max_len, gs.max_pages, G, gs.kv_pool.shape[-1],
                                           window), dtype=torch.uint8, device=DEV)
    freed = torch.full((U, gs.max_pages), -7, dtype=torch.int32, device=DEV)
    fcount = torch.full((U,), -7, dtype=torch.int32, device=DEV)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    se.se_snapkv_compact(_view(se, gs, hkv), G, qobs, window, kappa, scale, budget, max_len, flags,
                         freed, gs.max_pages, fcount, ws, err)
    torch.cuda.synchronize()
    return freed.cpu().numpy(), fcount.cpu().numpy(), se.se_read_device_errors(err)


def _compare(se, host, qobs_host, hkv, G, window, kappa, scale, budget, units=None, max_diverged=0):
    """Runs the library in score-only mode and in full on copies of `host` and
    compares every unit (or `units`) with the oracle.  Returns the number of
    units whose retained set differs from the oracle's by near-ties only."""
    U = host.lengths.numel()
    units = range(U) if units is None else units
    want = {}
    for u in units:
        st = oracle_unit(host, u)
        req, kvh = divmod(u, hkv)
        Qo = f64(qobs_host[req, :, kvh * G:(kvh + 1) * G, :])
        L = st.length
        before = {"K": st.K.copy(), "V": st.V.copy(), "pos": st.pos.copy(), "u": st.u.copy()}
        res = snapkv.compact_prompt(st, Qo, window, kappa, budget, scale)
        want[u] = (L, before, st, res)
    qobs = qobs_host.to(DEV)

    print(f"score-only U={U} G={G} w={window} kappa={kappa} B={budget}", flush=True)
    gs = to_device(host, DEV)
    _, fc0, err = _call(se, gs, hkv, G, qobs, window, kappa, scale, budget, se.SE_SNAPKV_SCORE_ONLY)
    assert err == 0
    assert torch.equal(gs.lengths.cpu(), host.lengths)
    for u in units:
        L, before, st, res = want[u]
        g = gpu_unit(gs, u)
        np.testing.assert_array_equal(g["pos"], before["pos"])
        np.testing.assert_array_equal(g["K"], before["K"])
        if L <= budget:
            np.testing.assert_array_equal(g["u"], before["u"])      # not touched
        else:
            assert_scores_close(g["u"], res["s"], f"unit {u} pooled scores")
            assert np.all(g["u"][L - window:] == 0.0)

    print("full", flush=True)
    gs = to_device(host, DEV)
    freed, fcount, err = _call(se, gs, hkv, G, qobs, window, kappa, scale, budget)
    assert err == 0
    bt = host.block_table.numpy()
    diverged = 0
    for u in units:
        L, before, st, res = want[u]
        assert int(gs.lengths[u]) == min(L, budget)
        g = gpu_unit(gs, u)
        if L <= budget:
            np.testing.assert_array_equal(g["pos"], before["pos"])
            np.testing.assert_array_equal(g["u"], before["u"])
            assert fcount[u] == 0
            continue
        kept_g, kept_o = set(g["pos"].tolist()), set(st.pos.tolist())
        if kept_g != kept_o:
            s_by_pos = dict(zip(before["pos"].tolist(), res["s"].tolist()))
            assert h2o_near_tie(s_by_pos, kept_g, kept_o), f"unit {u}: retained sets differ"
            # still a valid compaction: the window is kept and every slot holds an
            # original (position, key, value)
            assert set(before["pos"][L - window:].tolist()) <= kept_g
            row = {int(p): i for i, p in enumerate(before["pos"])}
            for i, p in enumerate(g["pos"]):
                np.testing.assert_array_equal(g["K"][i], before["K"][row[int(p)]])
                np.testing.assert_array_equal(g["V"][i], before["V"][row[int(p)]])
            diverged += 1
            continue
        np.testing.assert_array_equal(g["pos"], st.pos)
        np.testing.assert_array_equal(g["K"], st.K)
        np.testing.assert_array_equal(g["V"], st.V)
        assert_scores_close(g["u"], st.u, f"unit {u} scores after compaction")
        n = len(res["freed"])
        assert fcount[u] == n
        np.testing.assert_array_equal(freed[u, :n], bt[u, res["freed"]])
    assert diverged <= max_diverged, diverged
    return diverged


def test_scaled_workload_full_window(se):
    # the 8B head shape (G = 4, w = 32: 128 observation rows), ragged prompt
    # (1000 = 62.5 pages), heavy hitters, kappa 7
    w = scaled(SNAPKV, num_req=2, ctx=1000, budget=256)
    host = build_state(w, "cpu")
    qobs = build_observation(w, host, "cpu")
    _compare(se, host, qobs, w.hkv, w.q_per_kv, w.obs_window, w.pool_kernel, w.scale, w.budget,
             max_diverged=1)


@pytest.mark.parametrize("G,window,kappa,d,budget", [
    (4, 32, 7, 128, 256),    # 128 rows
    (4, 5, 3, 64, 100),      # 20 rows: a partial row tile
    (1, 64, 31, 128, 64),    # the window fills the budget; widest pooling
    (8, 16, 1, 128, 200),    # kappa 1: s = u
    (2, 7, 5, 64, 33),       # budget off the page size
])
def test_isolated_units(se, G, window, kappa, d, budget):
    hkv = 2
    lengths = [budget - 1, budget, budget + 1, 300, 777, 1601]
    host = isolated_units(lengths, max_pages=101, head_dim=d, seed=11 + G + window, num_kv_heads=hkv,
                          position_mode="contiguous")
    qobs = observation_queries(len(lengths) // hkv, window, hkv * G, d, seed=window)
    scale = float(np.float32(1.0 / np.sqrt(d)))
    _compare(se, host, qobs, hkv, G, window, kappa, scale, budget, max_diverged=1)


@pytest.mark.parametrize("G,window,kappa,d,budget", [
    (8, 32, 7, 128, 256),    # the paper's window with G = 8: 256 rows, two row blocks
    (4, 100, 5, 64, 160),    # 400 rows: four row blocks, the last one partial
    (2, 129, 3, 128, 300),   # 258 rows: a third block of two rows
])
def test_more_than_128_observation_rows(se, G, window, kappa, d, budget):
    # window x G above 128: row blocks of 128 rows score every key, the pool
    # kernel adds their partial sums in block order and pools
    hkv = 2
    lengths = [budget, budget + 1, 700, 1601]
    host = isolated_units(lengths, max_pages=101, head_dim=d, seed=3 + G + window, num_kv_heads=hkv,
                          position_mode="gapped")
    qobs = observation_queries(len(lengths) // hkv, window, hkv * G, d, seed=window + 1)
    scale = float(np.float32(1.0 / np.sqrt(d)))
    _compare(se, host, qobs, hkv, G, window, kappa, scale, budget, max_diverged=1)


def test_maximum_prompt_length(se):
    # one prompt at the call's maximum length (131072 slots, 8192 pages): the
    # eviction takes its streaming path for units this long
    host = isolated_units([131072], max_pages=8192, head_dim=128, seed=17, num_kv_heads=1,
                          position_mode="contiguous")
    qobs = observation_queries(1, 32, 4, 128, seed=18)
    _compare(se, host, qobs, 1, 4, 32, 7, float(np.float32(1 / np.sqrt(128))), 2048, max_diverged=1)


def test_gapped_positions(se):
    # sorted positions with gaps: a neighbourhood holds only the candidates within
    # kappa/2 positions, fewer than kappa/2 slots on a side
    lengths = [700, 1200]
    host = isolated_units(lengths, max_pages=80, head_dim=128, seed=5, num_kv_heads=1,
                          position_mode="gapped")
    qobs = observation_queries(2, 16, 4, 128, seed=6)
    _compare(se, host, qobs, 1, 4, 16, 9, float(np.float32(1 / np.sqrt(128))), 300, max_diverged=1)


@pytest.mark.parametrize("G,window", [(2, 8), (8, 40)])
def test_unsorted_positions_are_reported(se, G, window):
    lengths = [500]
    host = isolated_units(lengths, max_pages=40, head_dim=64, seed=8, num_kv_heads=1,
                          position_mode="shuffled")
    gs = to_device(host, DEV)
    qobs = observation_queries(1, window, G, 64, seed=9).to(DEV)
    _, _, err = _call(se, gs, 1, G, qobs, window, 3, 0.125, 100)
    assert err & se.SE_DEVERR_BAD_POSITIONS


def test_score_only_then_evict_equals_full(se):
    w = scaled(SNAPKV, num_req=2, ctx=900, budget=300)
    host = build_state(w, "cpu")
    qobs = build_observation(w, host, "cpu").to(DEV)
    a = to_device(host, DEV)
    _call(se, a, w.hkv, w.q_per_kv, qobs, w.obs_window, w.pool_kernel, w.scale, w.budget)
    b = to_device(host, DEV)
    _call(se, b, w.hkv, w.q_per_kv, qobs, w.obs_window, w.pool_kernel, w.scale, w.budget,
          se.SE_SNAPKV_SCORE_ONLY)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    se.se_evict_compact(_view(se, b, w.hkv), w.budget, w.obs_window, b.max_pages * 16, None, 0, None, err)
    torch.cuda.synchronize()
    assert se.se_read_device_errors(err) == 0
    assert torch.equal(a.lengths, b.lengths)
    for u in range(w.units_per_layer):
        ga, gb = gpu_unit(a, u), gpu_unit(b, u)
        for k in ("pos", "Kbits", "Vbits", "u"):
            np.testing.assert_array_equal(ga[k], gb[k])


def test_full_size_sampled_units(se):
    # the full 8B-shaped prompt compaction (64 requests x 8 KV heads x 32768
    # slots, w = 32, kappa = 7, B = 2048), as the benchmark times it; the oracle
    # checks sampled units one by one
    w = SNAPKV
    host_dev = build_state(w, DEV)
    qobs = build_observation(w, host_dev, DEV)
    sample = [0, 137, 511]
    sub = clone_state(host_dev)
    want = {}
    for u in sample:
        st = oracle_unit(host_dev, u)
        req, kvh = divmod(u, w.hkv)
        Qo = f64(qobs[req, :, kvh * w.q_per_kv:(kvh + 1) * w.q_per_kv, :])
        res = snapkv.compact_prompt(st, Qo, w.obs_window, w.pool_kernel, w.budget, w.scale)
        want[u] = (st, res)
    print("full-size score-only", flush=True)
    _, _, err = _call(se, sub, w.hkv, w.q_per_kv, qobs, w.obs_window, w.pool_kernel, w.scale, w.budget,
                      se.SE_SNAPKV_SCORE_ONLY)
    assert err == 0
    for u in sample:
        assert_scores_close(gpu_unit(sub, u)["u"], want[u][1]["s"], f"unit {u}")
    del sub
    print("full-size compaction", flush=True)
    _, _, err = _call(se, host_dev, w.hkv, w.q_per_kv, qobs, w.obs_window, w.pool_kernel, w.scale, w.budget)
    assert err == 0
    assert bool((host_dev.lengths == w.budget).all())
    for u in sample:
        st, res = want[u]
        g = gpu_unit(host_dev, u)
        kept_g, kept_o = set(g["pos"].tolist()), set(st.pos.tolist())
        if kept_g != kept_o:
            s_by_pos = dict(zip(range(w.ctx), res["s"].tolist()))
            assert h2o_near_tie(s_by_pos, kept_g, kept_o), f"unit {u}: retained sets differ"
            continue
        np.testing.assert_array_equal(g["pos"], st.pos)
        np.testing.assert_array_equal(g["K"], st.K)
        np.testing.assert_array_equal(g["V"], st.V)
