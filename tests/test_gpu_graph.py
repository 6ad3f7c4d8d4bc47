"""A layer-step's calls captured in a HIP graph (torch.cuda.graph) and replayed
give bit-identical results to the same calls run eagerly: every compute call
only enqueues kernels on the current stream, allocates nothing and never waits
for the device (the engine replays decode steps as graphs; Appendix B, "CUDA
Graph Execution").

Each test keeps two copies of one state.  The eager copy runs the calls
directly; the graph copy runs a graph captured once over static input
buffers, refilled before every replay.  Between replays the program does its
own eager work and synchronises; every replay is compared with its eager
counterpart.  The device error word is read outside the graph.
"""
import pytest
import torch

from workloads import LAYER_H2O, LAYER_QUEST, build_state, build_steps, clone_state, scaled

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
N_REPLAYS = 4


@pytest.fixture(scope="module")
def se():
    import paper_2609_39068_amd as m
    assert torch.cuda.is_available()
    return m


def _views(se, st):
    w = st.w
    return [se.KVView(st.kv_pool, st.pos_pool, st.score_pool, st.meta_pool, st.block_table[st.layer_rows(l)],
                      st.lengths[st.layer_rows(l)], num_kv_heads=w.hkv) for l in range(w.layers)]


def _static_inputs(steps, t):
    return [x.clone() for x in (steps.q[t], steps.k_new[t], steps.v_new[t], steps.new_pos[t])]


def test_h2o_layer_steps_replay_as_a_graph(se):
    # 3 layers of 512 units in the steady state (B = 2048, 2048 resident): each
    # replay runs se_decode_step_h2o on every layer (order kernel + attention
    # with the fused one-slot eviction), max_len = B + 1 as the scheduler passes it
    w = scaled(LAYER_H2O, layers=3, ctx=8192, initial_resident=2048, steps=N_REPLAYS)
    a = build_state(w, DEV)
    b = clone_state(a)
    steps = build_steps(w, a, DEV, steps=N_REPLAYS)
    U, G, d = w.units_per_layer, w.q_per_kv, w.head_dim
    ml = w.budget + 1
    assert int(a.lengths.max()) == w.budget

    def make(st):
        vs = _views(se, st)
        ws = se.H2ODecoder.workspace(vs[0], G, ml, DEV)
        err = torch.zeros(1, dtype=torch.int32, device=DEV)
        return [se.H2ODecoder(v, G, w.scale, w.budget, w.recent, ml, DEV, report_freed=True, ws=ws, dev_err=err)
                for v in vs]

    da, db = make(a), make(b)
    outs_a = [torch.empty((w.num_req, w.hq, d), dtype=torch.float32, device=DEV) for _ in range(w.layers)]
    outs_b = [torch.empty_like(o) for o in outs_a]
    lse_a = [torch.empty((w.num_req, w.hq), dtype=torch.float32, device=DEV) for _ in range(w.layers)]
    lse_b = [torch.empty_like(x) for x in lse_a]
    q, kn, vn, npos = _static_inputs(steps, 0)

    def layer_step(decs, outs, lses, q, kn, vn, npos):
        for l, dec in enumerate(decs):
            dec.step(q[l], kn[l], vn[l], npos, outs[l], lses[l], max_len=ml)

    # warm the library's kernels on a side stream before capture, on a scratch copy
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        c = clone_state(a)
        layer_step(make(c), [torch.empty_like(o) for o in outs_a], [torch.empty_like(x) for x in lse_a],
                   q, kn, vn, npos)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    del c

    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        layer_step(db, outs_b, lse_b, q, kn, vn, npos)
    torch.cuda.synchronize()
    for t in range(N_REPLAYS):
        print(f"replay {t}", flush=True)
        for dst, src in zip((q, kn, vn, npos), (steps.q[t], steps.k_new[t], steps.v_new[t], steps.new_pos[t])):
            dst.copy_(src)
        layer_step(da, outs_a, lse_a, steps.q[t], steps.k_new[t], steps.v_new[t], steps.new_pos[t])
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert se.se_read_device_errors(da[0].dev_err) == 0 and se.se_read_device_errors(db[0].dev_err) == 0
        for l in range(w.layers):
            assert torch.equal(outs_a[l], outs_b[l]) and torch.equal(lse_a[l], lse_b[l]), (t, l)
            assert torch.equal(da[l].freed_count, db[l].freed_count), (t, l)
        for name in ("kv_pool", "pos_pool", "score_pool", "lengths"):
            assert torch.equal(getattr(a, name), getattr(b, name)), (t, name)
        assert int(a.lengths.max()) == w.budget


def test_quest_layer_steps_replay_as_a_graph(se):
    # 256 units (one work-group each): se_decode_step_quest selects inside the
    # attention kernel; every replay appends one token per unit
    w = scaled(LAYER_QUEST, ctx=3001, top_k=16, steps=N_REPLAYS)
    a = build_state(w, DEV)
    b = clone_state(a)
    steps = build_steps(w, a, DEV, steps=N_REPLAYS)
    U, G, d = w.units_per_layer, w.q_per_kv, w.head_dim
    ml = a.max_pages * 16
    da = se.QuestDecoder(_views(se, a)[0], G, w.scale, w.top_k, ml, DEV)
    db = se.QuestDecoder(_views(se, b)[0], G, w.scale, w.top_k, ml, DEV)
    da.summarize()
    db.summarize()
    oa = torch.empty((w.num_req, w.hq, d), dtype=torch.float32, device=DEV)
    ob, la, lb = torch.empty_like(oa), torch.empty((w.num_req, w.hq), device=DEV), torch.empty((w.num_req, w.hq), device=DEV)
    q, kn, vn, npos = _static_inputs(steps, 0)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        db.step(q[0], kn[0], vn[0], npos, ob, lb)
    torch.cuda.synchronize()
    for t in range(N_REPLAYS):
        print(f"replay {t}", flush=True)
        for dst, src in zip((q, kn, vn, npos), (steps.q[t], steps.k_new[t], steps.v_new[t], steps.new_pos[t])):
            dst.copy_(src)
        da.step(steps.q[t, 0], steps.k_new[t, 0], steps.v_new[t, 0], steps.new_pos[t], oa, la)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert se.se_read_device_errors(da.dev_err) == 0 and se.se_read_device_errors(db.dev_err) == 0
        assert torch.equal(da.sel, db.sel), t
        assert torch.equal(oa, ob) and torch.equal(la, lb), t
        for name in ("kv_pool", "pos_pool", "meta_pool", "lengths"):
            assert torch.equal(getattr(a, name), getattr(b, name)), (t, name)
