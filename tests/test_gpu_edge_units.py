"""Units at the smallest sizes, on the GPU against the oracle: empty units,
one-slot units and units just under a page, mixed in one batch with ordinary
ones.

Closed forms pin the one-slot case without the oracle: softmax over a single
key is 1, so the output is that key's value row (up to float32 rounding of
w * v / w), the lse is its logit and its H2O score is G (one weight of 1 per
query head of the group); the Quest append of a key into a fresh page sets the
page's min and max to the key.
"""
import math

import numpy as np
import pytest
import torch

from oracle import h2o
from oracle.attention import selected_attention
from tests.oracle_bridge import LSE_ATOL, OUT_ATOL, assert_scores_close, f64, gpu_unit, oracle_unit
from workloads import isolated_units, to_device

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
G, D = 4, 128
SCALE = float(np.float32(1.0 / math.sqrt(D)))


@pytest.fixture(scope="module")
def se():
    import paper_2609_39068_amd as m
    assert torch.cuda.is_available()
    return m


def _view(se, st):
    return se.KVView(st.kv_pool, st.pos_pool, st.score_pool, st.meta_pool, st.block_table,
                     st.lengths, num_kv_heads=st.w.hkv)


def _token(U, seed):
    g = torch.Generator().manual_seed(seed)
    q = torch.randn((U, G, D), generator=g).to(torch.bfloat16)
    k = torch.randn((U, 1, D), generator=g).to(torch.bfloat16)
    v = torch.randn((U, 1, D), generator=g).to(torch.bfloat16)
    pos = torch.arange(U, dtype=torch.int32) + 90000      # above every resident position
    return q, k, v, pos


def test_h2o_step_on_empty_and_tiny_units(se):
    lengths = [0, 1, 37, 0, 15, 300]
    budget, recent, max_pages = 64, 8, 24
    host = isolated_units(lengths, max_pages, D, seed=41)
    gs = to_device(host, DEV)
    U = len(lengths)
    q, k, v, pos = _token(U, 5)
    dec = se.H2ODecoder(_view(se, gs), G, SCALE, budget, recent, max_pages * 16, DEV, report_freed=True)
    out = torch.full((U, G, D), float("nan"), dtype=torch.float32, device=DEV)
    lse = torch.full((U, G), float("nan"), dtype=torch.float32, device=DEV)
    dec.step(q.to(DEV), k.to(DEV), v.to(DEV), pos.to(DEV), out, lse)
    torch.cuda.synchronize()
    assert se.se_read_device_errors(dec.dev_err) == 0
    o_gpu, l_gpu = out.cpu().double().numpy(), lse.cpu().double().numpy()
    for u, L in enumerate(lengths):
        st = oracle_unit(host, u)
        res = h2o.decode_step(st, f64(q[u]), f64(k[u, 0]), f64(v[u, 0]), int(pos[u]), SCALE, budget, recent)
        assert np.abs(o_gpu[u] - res["o"]).max() <= OUT_ATOL
        assert np.abs(l_gpu[u] - res["lse"]).max() <= LSE_ATOL
        g = gpu_unit(gs, u)
        assert int(gs.lengths[u]) == min(L + 1, budget)
        np.testing.assert_array_equal(g["pos"], st.pos)
        np.testing.assert_array_equal(g["K"], st.K)
        np.testing.assert_array_equal(g["V"], st.V)
        assert_scores_close(g["u"], st.u, f"unit {u}")
        if L == 0:
            # one key: weight 1 per head, output = the value row, lse = the logit
            np.testing.assert_allclose(o_gpu[u], np.broadcast_to(f64(v[u, 0]), (G, D)), rtol=1e-6, atol=0)
            np.testing.assert_allclose(g["u"], [float(G)], rtol=1e-6, atol=0)
            z = (f64(q[u]) @ f64(k[u, 0])) * SCALE
            np.testing.assert_allclose(l_gpu[u], z, rtol=0, atol=1e-4)
    assert int(dec.freed_count[5]) == -(-301 // 16) - budget // 16


def test_attend_without_append_skips_empty_units(se):
    # With no append an empty unit has nothing to attend: its length is
    # reported as bad and its output rows are left as they were; the other
    # units of the batch are unaffected.
    lengths = [0, 1, 16, 0, 17]
    max_pages = 4
    host = isolated_units(lengths, max_pages, D, seed=43)
    gs = to_device(host, DEV)
    U = len(lengths)
    q, _, _, _ = _token(U, 7)
    max_len = max_pages * 16
    ws = torch.zeros(max(1, se.se_workspace_bytes(se.SE_OP_DECODE_ATTEND, U, max_len, max_pages, G, D)),
                     dtype=torch.uint8, device=DEV)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    out = torch.full((U, G, D), 7.0, dtype=torch.float32, device=DEV)
    lse = torch.full((U, G), 7.0, dtype=torch.float32, device=DEV)
    se.se_decode_attend(_view(se, gs), G, q.to(DEV), None, None, None, None, 0, SCALE, max_len,
                        se.SE_ATTEND_ACCUMULATE, out, lse, None, 0, ws, err)
    torch.cuda.synchronize()
    assert se.se_read_device_errors(err) == se.SE_DEVERR_BAD_LENGTH
    o_gpu, l_gpu = out.cpu().double().numpy(), lse.cpu().double().numpy()
    for u, L in enumerate(lengths):
        g = gpu_unit(gs, u)
        st = oracle_unit(host, u)
        assert int(gs.lengths[u]) == L
        if L == 0:
            assert (o_gpu[u] == 7.0).all() and (l_gpu[u] == 7.0).all()
            continue
        o, l, alpha, _ = selected_attention(f64(q[u]), st.K, st.V, np.arange(L), SCALE)
        assert np.abs(o_gpu[u] - o).max() <= OUT_ATOL
        assert np.abs(l_gpu[u] - l).max() <= LSE_ATOL
        assert_scores_close(g["u"], st.u + alpha.sum(axis=0), f"unit {u}")


def test_evict_compact_on_empty_and_tiny_units(se):
    # At or under the budget eviction changes nothing, empty units included.
    lengths = [0, 1, 0, 2]
    host = isolated_units(lengths, 2, D, seed=47, position_mode="shuffled")
    gs = to_device(host, DEV)
    before = [gpu_unit(gs, u) for u in range(len(lengths))]
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    cnt = torch.full((len(lengths),), -7, dtype=torch.int32, device=DEV)
    se.se_evict_compact(_view(se, gs), 1, 1, 32, None, 0, cnt, err)
    torch.cuda.synchronize()
    assert se.se_read_device_errors(err) == 0
    for u, L in enumerate(lengths):
        st = oracle_unit(host, u)
        keep = h2o.retain(st.pos, st.u, 1, 1)
        h2o.compact(st, keep, 1)
        g = gpu_unit(gs, u)
        assert int(gs.lengths[u]) == min(L, 1)
        np.testing.assert_array_equal(g["pos"], st.pos)
        np.testing.assert_array_equal(g["K"], st.K)
        if L <= 1:
            np.testing.assert_array_equal(g["pos"], before[u]["pos"])
        assert int(cnt[u]) == 0


@pytest.mark.parametrize("fused", [True, False])
def test_quest_step_on_units_within_one_page(se, fused):
    # Units whose whole cache is the current page: no candidate pages, so the
    # step attends every slot (dense attention); the append starts or extends
    # page 0's min/max.
    lengths = [0, 1, 14, 0]
    top_k, max_pages = 4, 4
    host = isolated_units(lengths, max_pages, D, seed=53, with_meta=True)
    gs = to_device(host, DEV)
    U = len(lengths)
    q, k, v, pos = _token(U, 11)
    view = _view(se, gs)
    dec = se.QuestDecoder(view, G, SCALE, top_k, max_pages * 16, DEV)
    dec.summarize()
    out = torch.full((U, G, D), float("nan"), dtype=torch.float32, device=DEV)
    lse = torch.full((U, G), float("nan"), dtype=torch.float32, device=DEV)
    dec.step(q.to(DEV), k.to(DEV), v.to(DEV), pos.to(DEV), out, lse, fused=fused)
    torch.cuda.synchronize()
    assert se.se_read_device_errors(dec.dev_err) == 0
    assert (dec.sel.cpu() == -1).all()
    o_gpu, l_gpu = out.cpu().double().numpy(), lse.cpu().double().numpy()
    meta = gs.meta_pool.cpu()
    for u, L in enumerate(lengths):
        st = oracle_unit(host, u)
        h2o.append(st, f64(k[u, 0]), f64(v[u, 0]), int(pos[u]))
        o, l, _, _ = selected_attention(f64(q[u]), st.K, st.V, np.arange(L + 1), SCALE)
        assert np.abs(o_gpu[u] - o).max() <= OUT_ATOL
        assert np.abs(l_gpu[u] - l).max() <= LSE_ATOL
        assert int(gs.lengths[u]) == L + 1
        page = int(host.block_table[u, 0])
        np.testing.assert_array_equal(f64(meta[page, 0]), st.K.min(axis=0))
        np.testing.assert_array_equal(f64(meta[page, 1]), st.K.max(axis=0))
        if L == 0:
            np.testing.assert_allclose(o_gpu[u], np.broadcast_to(f64(v[u, 0]), (G, D)), rtol=1e-6, atol=0)
