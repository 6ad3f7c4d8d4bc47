"""H2O chunk-wise prefill eviction on the GPU against the oracle:
se_h2o_prefill_chunk (the chunk's scores from its last queries, then H2O's
retention and compaction), one chunk and sequences of chunks.

Every chunk is checked by the same protocol as the decode steps: the oracle
starts from the GPU's state before the chunk; a copy of that state takes the
chunk with a budget no unit reaches (the call then only scores), which exposes
the GPU's fp32 scores before the retention; the oracle's scores must agree
with them (1e-3 relative), and the oracle's retention and compaction fed those
fp32 scores must give the real call's retained set, slot layout, K/V bits,
positions, scores and freed pages exactly.  The oracle's float64 retention may
differ from that only by swaps of near-tied slots.  No unit is dropped.

Every input comes from the seeded generators in workloads/.  The test writes
each chunk's keys, values and positions into the pools, as the prefill does
before calling.
"""
import numpy as np
import pytest
import torch

from oracle import h2o
from oracle.state import new_unit
from tests.oracle_bridge import assert_scores_close, f64, gpu_unit, h2o_near_tie, oracle_unit
from workloads import (H2O_PREFILL, build_observation, build_state, clone_state, isolated_units, observation_queries,
                       to_device)

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


@pytest.fixture(scope="module")
def se():
    import paper_2609_39068_amd as m
    assert torch.cuda.is_available()
    return m


def _view(se, st, hkv):
    return se.KVView(st.kv_pool, st.pos_pool, st.score_pool, None, st.block_table, st.lengths, num_kv_heads=hkv)


def _write_chunk(st, u, L0, K, V, pos):
    """The prefill's write of a chunk into unit u's slots [L0, L0 + C) (host tensors)."""
    for c in range(K.shape[0]):
        s = L0 + c
        ph = int(st.block_table[u, s // 16])
        st.kv_pool[ph, 0, s % 16] = K[c]
        st.kv_pool[ph, 1, s % 16] = V[c]
        st.pos_pool[ph, s % 16] = int(pos[c])
        st.score_pool[ph, s % 16] = 123.0            # stale: the call starts the chunk from 0
    st.lengths[u] = L0 + K.shape[0]


def _scored_copy(se, gs, hkv, G, qs, sw, C, scale, recent, max_len, ws, err):
    """A copy of the state after the chunk's scoring alone: with a budget of
    max_len no unit evicts, so its scores are the GPU's fp32 scores before the
    retention (the scoring does not depend on the budget)."""
    cs = clone_state(gs)
    se.se_h2o_prefill_chunk(_view(se, cs, hkv), G, qs, sw, C, scale, max_len, recent, max_len, None, 0, None, ws, err)
    return cs


def _check_chunk(where, r, c, g, budget, recent, fc, fp, bt_row):
    """One unit after one chunk.  r: the oracle's chunk from the GPU's
    pre-chunk state; c: the GPU unit after scoring only; g: after the real
    call; fc / fp / bt_row: its freed count, freed pages and block-table row.
    Returns 1 when the float64 retention differs from the fp32 one by near
    ties."""
    np.testing.assert_array_equal(c["pos"], r["pos_after_append"], err_msg=f"{where}: positions")
    assert_scores_close(c["u"], r["u_after_accumulate"], where)
    keep = h2o.retain(c["pos"], c["u"], budget, recent)
    st = new_unit(c["K"].copy(), c["V"].copy(), c["pos"].copy(), c["u"].copy())
    _, _, freed = h2o.compact(st, keep, budget)
    np.testing.assert_array_equal(g["pos"], st.pos, err_msg=f"{where}: retained positions")
    np.testing.assert_array_equal(g["K"], st.K, err_msg=f"{where}: keys")
    np.testing.assert_array_equal(g["V"], st.V, err_msg=f"{where}: values")
    np.testing.assert_array_equal(g["u"], st.u, err_msg=f"{where}: scores")
    assert fc == len(freed), f"{where}: freed count"
    np.testing.assert_array_equal(fp[:len(freed)], bt_row[freed], err_msg=f"{where}: freed pages")
    if np.array_equal(keep, r["keep"]):
        return 0
    by_pos = dict(zip(r["pos_after_append"].tolist(), r["u_after_accumulate"].tolist()))
    pos = c["pos"]
    assert h2o_near_tie(by_pos, set(pos[keep].tolist()), set(pos[r["keep"]].tolist())), \
        f"{where}: float64 retention differs beyond a near tie"
    return 1


def _run(se, lengths0, hkv, G, d, chunks, sw, budget, recent, seed):
    """Runs the chunks through every unit, each checked after every chunk by
    the protocol above.  Returns the number of near-tie differences."""
    U = len(lengths0)
    nreq = U // hkv
    cap = max(lengths0) + sum(chunks) + 16
    host = isolated_units(lengths0, -(-cap // 16), d, seed, num_kv_heads=hkv, position_mode="gapped")
    scale = float(np.float32(1 / np.sqrt(d)))
    gs = to_device(host, DEV)
    max_len = cap
    ws = torch.empty(se.se_workspace_bytes(se.SE_OP_H2O_PREFILL, U, max_len, host.max_pages, G, d, sw),
                     dtype=torch.uint8, device=DEV)
    freed = torch.full((U, host.max_pages), -7, dtype=torch.int32, device=DEV)
    fcount = torch.zeros(U, dtype=torch.int32, device=DEV)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    near = 0
    for ci, C in enumerate(chunks):
        kc = observation_queries(nreq, C, hkv, d, seed + 10 * ci + 1)
        vc = observation_queries(nreq, C, hkv, d, seed + 10 * ci + 2)
        qs = observation_queries(nreq, sw, hkv * G, d, seed + 10 * ci + 3)
        # the device state gathered to the host (the oracle starts from it), the
        # chunk written, and back
        hs = type(host)(**{**host.__dict__, "kv_pool": gs.kv_pool.cpu(), "pos_pool": gs.pos_pool.cpu(),
                           "score_pool": gs.score_pool.cpu(), "lengths": gs.lengths.cpu(),
                           "block_table": gs.block_table.cpu()})
        ost, cpos = {}, {}
        for u in range(U):
            req, h = divmod(u, hkv)
            L0 = int(hs.lengths[u])
            ost[u] = oracle_unit(hs, u)
            base = int(max(ost[u].pos.max() + 1, 0)) if ost[u].length else 0
            cpos[u] = base + 3 * np.arange(C)
            _write_chunk(hs, u, L0, kc[req, :, h], vc[req, :, h], cpos[u])
        gs = to_device(hs, DEV)
        print(f"chunk {ci}: C={C} sw={sw} G={G} d={d} B={budget} w={recent}", flush=True)
        cs = _scored_copy(se, gs, hkv, G, qs.to(DEV), sw, C, scale, recent, max_len, ws, err)
        se.se_h2o_prefill_chunk(_view(se, gs, hkv), G, qs.to(DEV), sw, C, scale, budget, recent, max_len, freed,
                                host.max_pages, fcount, ws, err)
        torch.cuda.synchronize()
        assert se.se_read_device_errors(err) == 0
        fc, fp = fcount.cpu().numpy(), freed.cpu().numpy()
        bt = hs.block_table.numpy()
        for u in range(U):
            req, h = divmod(u, hkv)
            r = h2o.prefill_chunk(ost[u], f64(kc[req, :, h]), f64(vc[req, :, h]), cpos[u],
                                  f64(qs[req, :, h * G:(h + 1) * G]), scale, budget, recent)
            near += _check_chunk(f"chunk {ci} unit {u}", r, gpu_unit(cs, u), gpu_unit(gs, u), budget, recent,
                                 fc[u], fp[u], bt[u])
    return near


@pytest.mark.parametrize("G,d,sw", [(4, 128, 32), (4, 128, 64), (2, 64, 100), (1, 128, 7), (8, 64, 16),
                                    (4, 128, 100), (8, 64, 40), (2, 128, 256), (1, 64, 257)])
def test_chunk_sequence(se, G, d, sw):
    # ragged retained states (an empty one among them), three chunks of 300,
    # 257 and 400 tokens, budget 512 with a 256-token window (ratio 0.5);
    # sw * G from 7 to 200 rows (two row blocks for 64 x 4 and 100 x 2), and
    # 257 to 512 rows, where one work-group holds every row and the unit's
    # pages are split over several (some parts of the short units are empty)
    lengths0 = [0, 0, 100, 100, 511, 511, 700, 700]
    _run(se, lengths0, 2, G, d, [300, 257, 400], sw, 512, 256, seed=G * 100 + sw)


def test_whole_chunk_scoring_without_eviction(se):
    # every query of the chunk scores (sw = C) and the budget holds everything:
    # each slot's accumulated score is compared
    _run(se, [50, 50, 200, 200], 2, 4, 64, [96], 96, 4096, 64, seed=3)


def test_short_chunk_behind_a_long_state(se):
    # a 16-token chunk after 3000 retained slots: one page of window keys
    _run(se, [3000, 3000], 2, 4, 128, [16, 33], 16, 2048, 1024, seed=8)


def test_length_below_chunk_is_reported(se):
    st = isolated_units([20, 20], 8, 64, 1, num_kv_heads=2)
    gs = to_device(st, DEV)
    view = _view(se, gs, 2)
    q = observation_queries(1, 4, 4, 64, 2).to(DEV)
    ws = torch.empty(se.se_workspace_bytes(se.SE_OP_H2O_PREFILL, 2, 128, 8, 2, 64, 4), dtype=torch.uint8, device=DEV)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    before = gs.score_pool.clone()
    se.se_h2o_prefill_chunk(view, 2, q, 4, 32, 0.125, 64, 4, 128, None, 0, None, ws, err)
    torch.cuda.synchronize()
    assert se.se_read_device_errors(err) & se.SE_DEVERR_BAD_LENGTH
    assert torch.equal(before, gs.score_pool)


def test_full_workload_sampled_units(se):
    # the 8B-shaped prefill workload at full size, in the launch configuration
    # the benchmark times (64 units of 2048 retained + 8192 chunk slots, 128
    # scoring queries x 4 heads = 4 row blocks, budget 2048, window 1024); the
    # oracle takes three sampled units from the same generated state
    w = H2O_PREFILL
    U, G, C, sw = w.units_per_layer, w.q_per_kv, w.chunk, w.obs_window
    gs = build_state(w, DEV)
    qs = build_observation(w, gs, DEV)
    sample = [0, 29, U - 1]
    ost = {}
    for u in sample:
        st = oracle_unit(gs, u)
        st.u[-C:] = 0.0                      # the chunk's stale scores: the call starts them at 0
        ost[u] = st
    bt = gs.block_table.cpu().numpy()
    max_len = gs.max_pages * 16
    ws = torch.empty(se.se_workspace_bytes(se.SE_OP_H2O_PREFILL, U, max_len, gs.max_pages, G, w.head_dim, sw),
                     dtype=torch.uint8, device=DEV)
    freed = torch.full((U, gs.max_pages), -7, dtype=torch.int32, device=DEV)
    fcount = torch.zeros(U, dtype=torch.int32, device=DEV)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    print(f"full prefill workload: U={U} L={int(gs.lengths[0])} C={C} sw={sw}", flush=True)
    cs = _scored_copy(se, gs, w.hkv, G, qs, sw, C, w.scale, w.recent, max_len, ws, err)
    se.se_h2o_prefill_chunk(_view(se, gs, w.hkv), G, qs, sw, C, w.scale, w.budget, w.recent, max_len, freed,
                            gs.max_pages, fcount, ws, err)
    torch.cuda.synchronize()
    assert se.se_read_device_errors(err) == 0
    assert bool((gs.lengths == w.budget).all())
    fc, fp = fcount.cpu().numpy(), freed.cpu().numpy()
    q = qs.cpu()
    for u in sample:
        req, h = divmod(u, w.hkv)
        r = h2o.chunk_eviction(ost[u], C, f64(q[req, :, h * G:(h + 1) * G]), w.scale, w.budget, w.recent)
        _check_chunk(f"unit {u}", r, gpu_unit(cs, u), gpu_unit(gs, u), w.budget, w.recent, fc[u], fp[u], bt[u])


def test_maximum_length(se):
    # a unit at the call's maximum length (131072 slots), its last 4096 slots the
    # chunk, scored by 16 queries of 4 heads; the eviction takes its streaming
    # path for a unit this long
    L, C, sw, G, d, budget, recent = 131072, 4096, 16, 4, 128, 2048, 1024
    host = isolated_units([L], 8192, d, 23, num_kv_heads=1, position_mode="contiguous")
    st = oracle_unit(host, 0)
    st.u[-C:] = 0.0                          # the chunk starts from 0
    qs = observation_queries(1, sw, G, d, 24)
    scale = float(np.float32(1 / np.sqrt(d)))
    gs = to_device(host, DEV)
    ws = torch.empty(se.se_workspace_bytes(se.SE_OP_H2O_PREFILL, 1, L, 8192, G, d, sw), dtype=torch.uint8,
                     device=DEV)
    freed = torch.full((1, 8192), -7, dtype=torch.int32, device=DEV)
    fcount = torch.zeros(1, dtype=torch.int32, device=DEV)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    print(f"maximum length: L={L} C={C} sw={sw}", flush=True)
    cs = _scored_copy(se, gs, 1, G, qs.to(DEV), sw, C, scale, recent, L, ws, err)
    se.se_h2o_prefill_chunk(_view(se, gs, 1), G, qs.to(DEV), sw, C, scale, budget, recent, L, freed, 8192, fcount,
                            ws, err)
    torch.cuda.synchronize()
    assert se.se_read_device_errors(err) == 0
    assert int(gs.lengths[0]) == budget
    r = h2o.chunk_eviction(st, C, f64(qs[0]), scale, budget, recent)
    _check_chunk("maximum length", r, gpu_unit(cs, 0), gpu_unit(gs, 0), budget, recent, int(fcount[0]),
                 freed[0].cpu().numpy(), host.block_table[0].numpy())

