"""H2O path on the GPU against the oracle: se_decode_step_h2o (append,
attention, fused score update and eviction) over whole trajectories,
se_decode_attend, se_accumulate_scores and se_evict_compact.

Every input comes from the seeded generators in workloads/.  Trajectories
follow the step protocol of tests/protocol.py: the oracle takes each step from
the GPU's pre-step state, and retention and compaction are compared bit for
bit on the GPU's own fp32 scores.
"""

import numpy as np
import pytest
import torch

from oracle import h2o
from oracle.attention import selected_attention
from tests.oracle_bridge import assert_scores_close, f64, gpu_unit, oracle_unit
from tests.protocol import h2o_trajectory
from workloads import (LAYER_H2O, TINY_H2O, build_state, build_steps, clone_state, isolated_units, scaled, step_bounds,
                       to_device)

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


@pytest.fixture(scope="module")
def se():
    import paper_2609_39068_amd as m
    assert torch.cuda.is_available()
    return m


def _view(se, st):
    return se.KVView(st.kv_pool, st.pos_pool, st.score_pool, st.meta_pool, st.block_table,
                     st.lengths, num_kv_heads=st.w.hkv)


def _run_h2o(se, w, n_steps):
    """n_steps fused H2O steps (se_decode_step_h2o with the benchmark's per-step
    max_len) on a device-generated workload, every unit checked against the
    oracle at every step (tests/protocol.py).  Returns unit-steps checked."""
    print(f"workload {w.name}: {w.units_per_layer} units, {n_steps} steps", flush=True)
    gs = build_state(w, DEV)
    steps = build_steps(w, gs, DEV, steps=n_steps)
    bounds = step_bounds(w, gs.lengths.cpu().tolist(), n_steps)
    checked, _ = h2o_trajectory(se, gs, steps, n_steps, {l: range(w.units_per_layer) for l in range(w.layers)},
                                q_per_kv=w.q_per_kv, scale=w.scale, budget=w.budget, recent=w.recent,
                                bounds=bounds, device=DEV)
    return checked


def test_tiny_h2o_step(se):
    w = TINY_H2O
    assert _run_h2o(se, w, 1) == w.units_per_layer


def test_trajectory_8b_shape_scaled(se):
    # 4 requests of the 8B head shape, a ragged initial context (1000 = 62.5
    # pages), budget 256 with a 32-token window: the first step takes the
    # general retention (1001 -> 256), the rest the steady one-slot path.
    w = scaled(LAYER_H2O, num_req=4, ctx=1000, budget=256, recent=32, steps=20)
    assert _run_h2o(se, w, 20) == 20 * w.units_per_layer


def test_trajectory_small_window_long_run(se):
    # d=64, G=2, budget not a multiple of the page size, window of 3.
    w = scaled(TINY_H2O, num_req=3, hq=4, hkv=2, ctx=150, budget=100, recent=3, steps=40)
    assert _run_h2o(se, w, 40) == 40 * w.units_per_layer


@pytest.mark.parametrize("G,d", [(1, 128), (2, 64), (4, 64), (8, 128), (8, 64)])
def test_head_group_and_dim_variants(se, G, d):
    w = scaled(TINY_H2O, num_req=2, hq=2 * G, hkv=2, head_dim=d, ctx=300, budget=64, recent=16, steps=3)
    assert _run_h2o(se, w, 3) == 3 * w.units_per_layer


@pytest.mark.parametrize("num_req,ctx,budget,recent", [(4, 3000, 2048, 256), (64, 2000, 1024, 128)])
def test_group_of_8_trajectory(se, num_req, ctx, budget, recent):
    # Groups of 8 query heads per KV head (two passes of the four-head
    # reduction): 32 units split over work-groups with a combine pass, and 512
    # units streamed whole with the fused eviction; the first step evicts down
    # to the budget, the rest are steady.
    w = scaled(LAYER_H2O, num_req=num_req, hq=64, hkv=8, ctx=ctx, budget=budget, recent=recent, steps=4)
    assert w.q_per_kv == 8
    assert _run_h2o(se, w, 4) == 4 * w.units_per_layer


def test_budget_covers_context_is_dense(se):
    # B >= L: TopK keeps everything (no eviction) and attention is dense.
    w = scaled(LAYER_H2O, num_req=2, ctx=200, budget=400, recent=8, steps=3)
    assert _run_h2o(se, w, 3) == 3 * w.units_per_layer


def test_unfused_accumulate_matches_fused(se):
    w = scaled(LAYER_H2O, num_req=2, ctx=700, budget=2048, recent=8, steps=1)
    host = build_state(w, "cpu")
    steps = build_steps(w, host, "cpu")
    a, b = to_device(host, DEV), to_device(host, DEV)
    va, vb = _view(se, a), _view(se, b)
    max_len = host.max_pages * 16
    G, U = w.q_per_kv, w.units_per_layer
    ws = torch.zeros(se.se_workspace_bytes(se.SE_OP_DECODE_ATTEND, U, max_len, host.max_pages, G, w.head_dim),
                     dtype=torch.uint8, device=DEV)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    out_a = torch.empty((w.num_req, w.hq, w.head_dim), dtype=torch.float32, device=DEV)
    out_b, lse_b = torch.empty_like(out_a), torch.empty((w.num_req, w.hq), dtype=torch.float32, device=DEV)
    logits = torch.full((U, G, max_len), float("nan"), dtype=torch.float32, device=DEV)
    args = (steps.q[0, 0].to(DEV), steps.k_new[0, 0].to(DEV), steps.v_new[0, 0].to(DEV), steps.new_pos[0].to(DEV))
    se.se_decode_attend(va, G, *args, None, 0, w.scale, max_len, se.SE_ATTEND_ACCUMULATE, out_a, None,
                        None, 0, ws, err)
    se.se_decode_attend(vb, G, *args, None, 0, w.scale, max_len, 0, out_b, lse_b, logits, max_len, ws, err)
    se.se_accumulate_scores(vb, G, logits, max_len, lse_b, max_len, err)
    torch.cuda.synchronize()
    assert se.se_read_device_errors(err) == 0
    assert torch.equal(out_a, out_b)
    for u in range(U):
        ga, gb = gpu_unit(a, u), gpu_unit(b, u)
        assert_scores_close(gb["u"], ga["u"], f"unit {u}")
        # logits are the scaled dot products of the oracle
        st = oracle_unit(host, u)
        req, kvh = divmod(u, w.hkv)
        h2o.append(st, f64(steps.k_new[0, 0, req, kvh]), f64(steps.v_new[0, 0, req, kvh]), 0)
        _, _, _, z = selected_attention(f64(steps.q[0, 0, req, kvh * G:(kvh + 1) * G]), st.K, st.V,
                                        np.arange(st.length), w.scale)
        np.testing.assert_allclose(logits[u, :, :st.length].cpu().double().numpy(), z, atol=1e-4, rtol=1e-5)


CASES = [
    # lengths, budget, recent, positions, score levels
    ([40, 17, 64], 64, 8, "contiguous", 0),          # L <= B everywhere: nothing changes
    ([65, 65, 65, 65], 64, 8, "contiguous", 0),      # steady state, one slot over
    ([65, 65, 65, 65], 64, 8, "shuffled", 3),        # steady, scattered window, many ties
    ([129, 129], 128, 0, "contiguous", 4),           # no window
    ([300, 257, 1000, 64], 64, 16, "contiguous", 0), # general radix path
    ([300, 257, 1000], 64, 16, "gapped", 5),         # window by radix over positions, ties
    ([300, 333], 100, 7, "shuffled", 2),             # budget off the page grid, two score levels
    ([90, 200], 40, 40, "shuffled", 0),              # window fills the budget
    ([90, 200], 40, 80, "contiguous", 0),            # window larger than the budget
    ([5000, 4097, 8000], 4096, 512, "shuffled", 0),  # the 8B budget
    ([4097] * 6, 4096, 512, "contiguous", 1000),     # steady at the 8B budget, ties
    ([32769, 20000], 2048, 256, "contiguous", 0),    # first step of the 8B workload
    ([6000, 3000], 1024, 64, "contiguous", 3),       # exact score ties at the threshold
    ([6000, 3000], 1024, 64, "shuffled", 1500),      # small tie classes (a few slots) at the threshold
    ([2000, 1500], 512, 32, "gapped", 40),           # tie classes of up to about 60 slots
    ([36000], 2048, 256, "shuffled", 7),             # past the register-resident size
    ([8193, 12000], 8192, 512, "shuffled", 0),       # the largest budget
    ([3, 1, 2, 0], 1, 1, "gapped", 2),               # budget 1: only the newest position stays
]


@pytest.mark.parametrize("d", [128, 64])
@pytest.mark.parametrize("lengths,budget,recent,mode,levels", CASES)
def test_evict_compact_bitexact(se, d, lengths, budget, recent, mode, levels):
    # The oracle selects on the same float32 scores the GPU holds, so retained
    # sets, the compacted layout and the freed pages must agree bit for bit.
    max_pages = -(-max(max(lengths), budget + 1) // 16)
    host = isolated_units(lengths, max_pages, d, seed=sum(lengths) + budget + recent + d,
                          position_mode=mode, score_levels=levels)
    gs = to_device(host, DEV)
    view = _view(se, gs)
    U = len(lengths)
    freed = torch.full((U, max_pages), -7, dtype=torch.int32, device=DEV)
    cnt = torch.full((U,), -7, dtype=torch.int32, device=DEV)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    se.se_evict_compact(view, budget, recent, max_pages * 16, freed, max_pages, cnt, err)
    torch.cuda.synchronize()
    assert se.se_read_device_errors(err) == 0
    for u, L in enumerate(lengths):
        st = oracle_unit(host, u)
        keep = h2o.retain(st.pos, st.u, budget, recent)
        _, _, fr = h2o.compact(st, keep, budget)
        g = gpu_unit(gs, u)
        assert int(gs.lengths[u]) == min(L, budget)
        np.testing.assert_array_equal(g["pos"], st.pos)
        np.testing.assert_array_equal(g["K"], st.K)
        np.testing.assert_array_equal(g["V"], st.V)
        np.testing.assert_array_equal(g["u"].astype(np.float32), st.u.astype(np.float32))
        assert int(cnt[u]) == len(fr)
        np.testing.assert_array_equal(freed[u, :len(fr)].cpu().numpy(), host.block_table[u, fr].numpy())


def test_device_errors_are_reported(se):
    # A block-table entry outside the pool, and a length above max_len, are
    # found on the device: the bit is set, the unit is skipped, nothing faults.
    host = isolated_units([100, 100], 8, 128, seed=5)
    bt = host.block_table.clone()
    bt[1, 2] = -1
    host.block_table = bt
    gs = to_device(host, DEV)
    view = _view(se, gs)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    se.se_evict_compact(view, 64, 8, 128, None, 0, None, err)
    torch.cuda.synchronize()
    assert se.se_read_device_errors(err) == se.SE_DEVERR_BAD_PAGE
    assert int(gs.lengths[0]) == 64 and int(gs.lengths[1]) == 100
    se.se_evict_compact(view, 64, 8, 80, None, 0, None, err)  # lengths above max_len
    torch.cuda.synchronize()
    assert se.se_read_device_errors(err) == se.SE_DEVERR_BAD_LENGTH
    # attention over a unit whose length is above max_len
    G, d = 4, 128
    q = torch.zeros((2, G, d), dtype=torch.bfloat16, device=DEV)
    out = torch.zeros((2, G, d), dtype=torch.float32, device=DEV)
    ws = torch.zeros(se.se_workspace_bytes(se.SE_OP_DECODE_ATTEND, 2, 32, 8, G, d), dtype=torch.uint8, device=DEV)
    se.se_decode_attend(view, G, q, None, None, None, None, 0, 0.1, 32, 0, out, None, None, 0, ws, err)
    torch.cuda.synchronize()
    assert se.se_read_device_errors(err) & se.SE_DEVERR_BAD_LENGTH
    assert float(out.abs().max()) == 0.0


def test_deterministic_and_resumable(se):
    # Two runs from the same state give bit-identical results, and a run that
    # is snapshotted and restored midway continues bit-identically.
    w = scaled(LAYER_H2O, num_req=2, ctx=600, budget=128, recent=16, steps=6)
    host = build_state(w, "cpu")
    steps = build_steps(w, host, "cpu")
    max_len = host.max_pages * 16

    def run(st, t0, t1):
        view = _view(se, st)
        dec = se.H2ODecoder(view, w.q_per_kv, w.scale, w.budget, w.recent, max_len, DEV)
        out = torch.empty((w.num_req, w.hq, w.head_dim), dtype=torch.float32, device=DEV)
        outs = []
        for t in range(t0, t1):
            dec.step(steps.q[t, 0].to(DEV), steps.k_new[t, 0].to(DEV), steps.v_new[t, 0].to(DEV),
                     steps.new_pos[t].to(DEV), out)
            outs.append(out.clone())
        torch.cuda.synchronize()
        return outs

    a, b = to_device(host, DEV), to_device(host, DEV)
    oa, ob = run(a, 0, 6), run(b, 0, 6)
    for x, y in zip(oa, ob):
        assert torch.equal(x, y)
    for name in ("kv_pool", "pos_pool", "score_pool", "lengths"):
        assert torch.equal(getattr(a, name), getattr(b, name))
    c = to_device(host, DEV)
    run(c, 0, 3)
    snap = clone_state(c)
    oc = run(snap, 3, 6)
    for x, y in zip(oa[3:], oc):
        assert torch.equal(x, y)
    for name in ("kv_pool", "pos_pool", "score_pool", "lengths"):
        assert torch.equal(getattr(a, name), getattr(snap, name))


FUSED_CASES = [
    # lengths, budget, window, block-table row length
    ([300, 129, 129, 129, 64, 128], 128, 16, 32),
    ([8193, 8192, 9000, 8192], 8192, 512, 570),   # the largest budget: long units, weights past LDS
    ([2, 1, 5, 0], 1, 1, 2),                      # budget 1: the window is the newest slot
]


@pytest.mark.parametrize("mode", ["contiguous", "gapped", "shuffled"])
@pytest.mark.parametrize("lengths,B,w,P", FUSED_CASES)
def test_fused_step_equals_attend_then_evict(se, mode, lengths, B, w, P):
    # se_decode_step_h2o must leave exactly the state that se_decode_attend +
    # se_evict_compact leave: bit-identical pools, lengths, outputs and freed
    # pages, whether the eviction is fused (steady, contiguous window) or not
    # (first step, or scattered recent positions).
    d, G = 128, 4
    host = isolated_units(lengths, P, d, seed=77 + B, num_kv_heads=2, position_mode=mode)
    U = len(lengths)
    nreq = U // 2
    g = torch.Generator().manual_seed(3)
    a, b = to_device(host, DEV), to_device(host, DEV)
    max_len = P * 16
    ws = torch.zeros(se.se_workspace_bytes(se.SE_OP_DECODE_ATTEND, U, max_len, P, G, d), dtype=torch.uint8, device=DEV)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    fa = torch.full((U, P), -3, dtype=torch.int32, device=DEV)
    fb = fa.clone()
    ca = torch.full((U,), -3, dtype=torch.int32, device=DEV)
    cb = ca.clone()
    va, vb = _view(se, a), _view(se, b)
    for step in range(4):
        q = torch.randn((nreq, 2 * G, d), generator=g).to(torch.bfloat16).to(DEV)
        kn = torch.randn((nreq, 2, d), generator=g).to(torch.bfloat16).to(DEV)
        vn = torch.randn((nreq, 2, d), generator=g).to(torch.bfloat16).to(DEV)
        npos = torch.tensor([1_000_000 + 10 * step + r for r in range(nreq)], dtype=torch.int32, device=DEV)
        oa = torch.empty((nreq, 2 * G, d), dtype=torch.float32, device=DEV)
        ob = torch.empty_like(oa)
        se.se_decode_attend(va, G, q, kn, vn, npos, None, 0, 0.088, max_len, se.SE_ATTEND_ACCUMULATE, oa,
                            None, None, 0, ws, err)
        se.se_evict_compact(va, B, w, max_len, fa, P, ca, err)
        se.se_decode_step_h2o(vb, G, q, kn, vn, npos, 0.088, B, w, max_len, ob, None, fb, P, cb, ws, err)
        torch.cuda.synchronize()
        assert se.se_read_device_errors(err) == 0
        assert torch.equal(oa, ob)
        for name in ("kv_pool", "pos_pool", "score_pool", "lengths"):
            assert torch.equal(getattr(a, name), getattr(b, name)), (step, name)
        assert torch.equal(ca, cb), step
        for u in range(U):
            n = int(ca[u])
            assert torch.equal(fa[u, :n], fb[u, :n])
