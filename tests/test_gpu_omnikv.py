"""OmniKV on the GPU against the oracle: an observation layer's step
(se_decode_attend with logits, then se_omnikv_select) and a sparse layer's
step over the selection (se_attend_slots).

Every input comes from the seeded generators in workloads/; the oracle reads
them before any library call touches them.  Where the sparse layer is checked
on its own, it is fed the oracle's selection (an oracle output as a library
input, never the reverse).
"""
import numpy as np
import pytest
import torch

from oracle import omnikv
from tests.oracle_bridge import LSE_ATOL, NEAR_TIE, OUT_ATOL, f64, oracle_unit
from workloads import isolated_units, observation_queries, to_device

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


@pytest.fixture(scope="module")
def se():
    import paper_2609_39068_amd as m
    assert torch.cuda.is_available()
    return m


def _view(se, st, hkv):
    return se.KVView(st.kv_pool, st.pos_pool, None, None, st.block_table, st.lengths, num_kv_heads=hkv)


def _inputs(nreq, hkv, G, d, seed):
    q = observation_queries(nreq, 1, hkv * G, d, seed)[:, 0].contiguous()
    k = observation_queries(nreq, 1, hkv, d, seed + 1)[:, 0].contiguous()
    v = observation_queries(nreq, 1, hkv, d, seed + 2)[:, 0].contiguous()
    return q, k, v


def _near_tie_sets(s, got, want):
    only_g, only_o = set(got) - set(want), set(want) - set(got)
    if len(only_g) != len(only_o):
        return False
    return all(s[y] - s[x] <= NEAR_TIE * max(1.0, abs(s[x]), abs(s[y])) for x in only_g for y in only_o)


def _run_step(se, ctx, hkv, G, d, budget, seed):
    """One decode step: observation layer A (dense attention + selection) and a
    sparse layer B (attention over A's selection), GPU against oracle.  The
    observation layer's logits (fp32, as the GPU formed them) must match the
    oracle's, and the oracle's TopK over their maximum over the request's heads
    must equal the GPU's selection exactly; the oracle's float64 selection may
    differ from it only by near ties.  Returns the number of requests whose
    float64 selection differs."""
    lengths = [L for L in ctx for _ in range(hkv)]
    nreq = len(ctx)
    max_pages = -(-(max(ctx) + 1) // 16) + 1
    A = isolated_units(lengths, max_pages, d, seed, num_kv_heads=hkv, position_mode="contiguous")
    B = isolated_units(lengths, max_pages, d, seed + 100, num_kv_heads=hkv, position_mode="contiguous")
    qa, ka, va = _inputs(nreq, hkv, G, d, seed)
    qb, kb, vb = _inputs(nreq, hkv, G, d, seed + 10)
    npos = torch.tensor([L for L in ctx], dtype=torch.int32)
    scale = float(np.float32(1 / np.sqrt(d)))
    # oracle, from the generator's tensors
    want = []
    for r in range(nreq):
        ua = [oracle_unit(A, r * hkv + h) for h in range(hkv)]
        ub = [oracle_unit(B, r * hkv + h) for h in range(hkv)]
        fa = omnikv.filter_step(ua, f64(qa[r]), f64(ka[r]), f64(va[r]), ctx[r], scale, budget)
        sb = omnikv.sparse_step(ub, f64(qb[r]), f64(kb[r]), f64(vb[r]), ctx[r], scale, fa["J"])
        want.append((fa, sb))
    # library
    ga, gb = to_device(A, DEV), to_device(B, DEV)
    va_, vb_ = _view(se, ga, hkv), _view(se, gb, hkv)
    U = nreq * hkv
    max_len = max(ctx) + 1
    stride = -(-max_len // 64) * 64
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    logits = torch.empty(U * G * stride, dtype=torch.float32, device=DEV)
    out_a = torch.empty((nreq, hkv * G, d), dtype=torch.float32, device=DEV)
    lse_a = torch.empty((nreq, hkv * G), dtype=torch.float32, device=DEV)
    ws = torch.empty(se.se_workspace_bytes(se.SE_OP_DECODE_ATTEND, U, max_len, ga.max_pages, G, d, 0),
                     dtype=torch.uint8, device=DEV)
    print(f"observation layer ctx={ctx} hkv={hkv} G={G} d={d} b={budget}", flush=True)
    se.se_decode_attend(va_, G, qa.to(DEV), ka.to(DEV), va.to(DEV), npos.to(DEV), None, 0, scale, max_len, 0,
                        out_a, lse_a, logits, stride, ws, err)
    sel = torch.full((nreq, budget), -7, dtype=torch.int32, device=DEV)
    ws2 = torch.empty(se.se_workspace_bytes(se.SE_OP_OMNIKV_SELECT, nreq, max_len, ga.max_pages, G, d, 0),
                      dtype=torch.uint8, device=DEV)
    se.se_omnikv_select(va_, G, logits, stride, budget, max_len, sel, ws2, err)
    torch.cuda.synchronize()
    assert se.se_read_device_errors(err) == 0
    sel_h = sel.cpu().numpy()
    o_a = out_a.cpu().double().numpy()
    lg = logits.cpu().numpy().astype(np.float64).reshape(nreq, hkv * G, stride)
    near = 0
    for r in range(nreq):
        fa, _ = want[r]
        assert np.abs(o_a[r] - fa["o"]).max() <= OUT_ATOL
        n_av = ctx[r] + 1                    # slots after the append
        s32 = lg[r, :, :n_av].max(axis=0)    # the GPU's fp32 scores, max over the request's heads
        rel = np.abs(s32 - fa["s"]) / np.maximum(1.0, np.abs(fa["s"]))
        assert rel.max() <= 1e-4, f"request {r}: scores off by {rel.max():.2e}"
        got = sel_h[r][sel_h[r] >= 0]
        n = min(budget, n_av)
        assert len(got) == n and np.all(np.diff(got) > 0)
        assert np.all(sel_h[r][n:] == -1)
        np.testing.assert_array_equal(got, omnikv.select(s32, budget), err_msg=f"request {r}: selection")
        if not np.array_equal(got, fa["J"]):
            assert _near_tie_sets(fa["s"], got.tolist(), fa["J"].tolist()), f"request {r}: selections differ"
            near += 1
    # sparse layer fed the oracle's selection
    Jo = torch.full((nreq, budget), -1, dtype=torch.int32)
    for r in range(nreq):
        Jo[r, :len(want[r][0]["J"])] = torch.from_numpy(want[r][0]["J"].astype(np.int32))
    out_b = torch.empty((nreq, hkv * G, d), dtype=torch.float32, device=DEV)
    lse_b = torch.empty((nreq, hkv * G), dtype=torch.float32, device=DEV)
    print("sparse layer", flush=True)
    se.se_attend_slots(vb_, G, qb.to(DEV), kb.to(DEV), vb.to(DEV), npos.to(DEV), Jo.to(DEV), budget, scale, max_len,
                       out_b, lse_b, err)
    torch.cuda.synchronize()
    assert se.se_read_device_errors(err) == 0
    o_b, l_b = out_b.cpu().double().numpy(), lse_b.cpu().double().numpy()
    for r in range(nreq):
        _, sb = want[r]
        assert np.abs(o_b[r] - sb["o"]).max() <= OUT_ATOL
        assert np.abs(l_b[r] - sb["lse"]).max() <= LSE_ATOL
    assert torch.equal(gb.lengths.cpu(), torch.tensor(lengths, dtype=torch.int32) + 1)
    return near


@pytest.mark.parametrize("ctx,hkv,G,d,budget", [
    ([300, 777, 1601], 2, 4, 128, 256),     # 8B-like group, ragged contexts, budget off the page size
    ([2000, 513], 2, 2, 128, 100),
    ([900, 1500], 4, 2, 64, 333),
    ([40, 700], 2, 1, 64, 64),               # the first request selects everything (padding)
])
def test_observation_then_sparse_layer(se, ctx, hkv, G, d, budget):
    _run_step(se, ctx, hkv, G, d, budget, seed=sum(ctx) + G)


def test_long_context_selection_from_workspace(se):
    # more slots than the selection keeps in LDS: the scores are ranked from the workspace
    _run_step(se, [40000], 1, 4, 128, 2048, seed=4)


@pytest.mark.parametrize("G,L,stride,budget", [(4, 1000, 1024, 97), (4, 1000, 1027, 97), (3, 1001, 1024, 97),
                                               (5, 999, 1000, 97), (4, 20000, 20000, 2048), (4, 36000, 36003, 2048),
                                               (4, 30001, 30004, 2048), (4, 40000, 40000, 2048),
                                               (2, 70000, 70000, 4096)])
def test_select_from_given_logits_with_ties(se, G, L, stride, budget):
    # logits taken as given (integer levels, many exact ties): the selection is
    # bit-exact against the oracle's TopK over max-over-heads scores; rows in
    # 16-byte aligned strides (four slots per load, 8 / 6 / 10 rows per request)
    # and unaligned strides; from 20000 slots on, every thread of the ranking
    # owns a run of 20 to 69 slots (the tie classes span many runs; at 30001 the
    # last run holds one slot), from 36865 on the scores are ranked from the
    # workspace
    hkv, nreq = 2, 3
    g = torch.Generator().manual_seed(5 + G + stride)
    logits = torch.randint(0, 7, (nreq * hkv * G, stride), generator=g).to(torch.float32)
    st = isolated_units([L] * (nreq * hkv), (L + 15) // 16, 64, 1, num_kv_heads=hkv, with_scores=False)
    gs = to_device(st, DEV)
    view = _view(se, gs, hkv)
    sel = torch.empty((nreq, budget), dtype=torch.int32, device=DEV)
    ws = torch.empty(se.se_workspace_bytes(se.SE_OP_OMNIKV_SELECT, nreq, L, (L + 15) // 16, G, 64, 0),
                     dtype=torch.uint8, device=DEV)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    se.se_omnikv_select(view, G, logits.to(DEV), stride, budget, L, sel, ws, err)
    torch.cuda.synchronize()
    assert se.se_read_device_errors(err) == 0
    lg = logits.numpy().astype(np.float64).reshape(nreq, hkv * G, stride)[:, :, :L]
    for r in range(nreq):
        J = omnikv.select(lg[r].max(axis=0), budget)
        np.testing.assert_array_equal(sel.cpu().numpy()[r], J)


def test_unequal_lengths_in_a_request_are_reported(se):
    hkv, G, L = 2, 2, 300
    st = isolated_units([L, L + 5], 32, 64, 2, num_kv_heads=hkv)
    gs = to_device(st, DEV)
    view = _view(se, gs, hkv)
    stride = 320
    logits = torch.zeros(hkv * G * stride, dtype=torch.float32, device=DEV)
    sel = torch.zeros((1, 16), dtype=torch.int32, device=DEV)
    ws = torch.empty(se.se_workspace_bytes(se.SE_OP_OMNIKV_SELECT, 1, stride, 32, G, 64, 0), dtype=torch.uint8,
                     device=DEV)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    se.se_omnikv_select(view, G, logits, stride, 16, stride, sel, ws, err)
    torch.cuda.synchronize()
    assert se.se_read_device_errors(err) & se.SE_DEVERR_BAD_LENGTH
    assert bool((sel == -1).all())


def test_attend_slots_edge_cases(se):
    # padding, the appended token, an out-of-range entry (reported, skipped) and an
    # empty selection
    hkv, G, d, L = 2, 4, 128, 500
    st = isolated_units([L, L, L, L], 40, d, 7, num_kv_heads=hkv)
    q, k, v = _inputs(2, hkv, G, d, 17)
    npos = torch.tensor([L, L], dtype=torch.int32)
    sel = torch.full((2, 8), -1, dtype=torch.int32)
    sel[0, :5] = torch.tensor([0, 17, 255, 499, L])          # L: the token appended now
    scale = float(np.float32(1 / np.sqrt(d)))
    units = [oracle_unit(st, u) for u in range(4)]
    res = omnikv.sparse_step(units[:2], f64(q[0]), f64(k[0]), f64(v[0]), L, scale, sel[0, :5].numpy())
    gs = to_device(st, DEV)
    view = _view(se, gs, hkv)
    out = torch.empty((2, hkv * G, d), dtype=torch.float32, device=DEV)
    lse = torch.empty((2, hkv * G), dtype=torch.float32, device=DEV)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    se.se_attend_slots(view, G, q.to(DEV), k.to(DEV), v.to(DEV), npos.to(DEV), sel.to(DEV), 8, scale, L + 1,
                       out, lse, err)
    torch.cuda.synchronize()
    assert se.se_read_device_errors(err) == 0
    assert np.abs(out.cpu().double().numpy()[0] - res["o"]).max() <= OUT_ATOL
    assert bool((out[1] == 0).all()) and bool(torch.isinf(lse[1]).all())
    bad = sel.clone()
    bad[1, 0] = L + 3
    se.se_attend_slots(view, G, q.to(DEV), None, None, None, bad.to(DEV), 8, scale, L + 1, out, lse, err)
    torch.cuda.synchronize()
    assert se.se_read_device_errors(err) & se.SE_DEVERR_BAD_SELECTION


@pytest.mark.parametrize("G,d,nreq", [
    (8, 128, 2), (8, 64, 2), (1, 128, 2), (4, 64, 2), (2, 64, 3),
    (4, 128, 130),   # 260 units: more than one work-group per compute unit (512 threads, not 1024)
])
def test_attend_slots_group_sizes(se, G, d, nreq):
    # a sparse layer over a fixed selection (every third slot and the new token)
    hkv, L = 2, 777
    st = isolated_units([L] * (nreq * hkv), 50, d, 9 + G, num_kv_heads=hkv)
    q, k, v = _inputs(nreq, hkv, G, d, 31 + G)
    npos = torch.full((nreq,), L, dtype=torch.int32)
    J = np.concatenate([np.arange(0, L, 3), [L]]).astype(np.int32)
    sel = torch.from_numpy(np.stack([J] * nreq))
    scale = float(np.float32(1 / np.sqrt(d)))
    want = []
    for r in range(nreq):
        units = [oracle_unit(st, r * hkv + h) for h in range(hkv)]
        want.append(omnikv.sparse_step(units, f64(q[r]), f64(k[r]), f64(v[r]), L, scale, J))
    gs = to_device(st, DEV)
    view = _view(se, gs, hkv)
    out = torch.empty((nreq, hkv * G, d), dtype=torch.float32, device=DEV)
    lse = torch.empty((nreq, hkv * G), dtype=torch.float32, device=DEV)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    se.se_attend_slots(view, G, q.to(DEV), k.to(DEV), v.to(DEV), npos.to(DEV), sel.to(DEV), len(J), scale, L + 1,
                       out, lse, err)
    torch.cuda.synchronize()
    assert se.se_read_device_errors(err) == 0
    for r in range(nreq):
        assert np.abs(out.cpu().double().numpy()[r] - want[r]["o"]).max() <= OUT_ATOL
        assert np.abs(lse.cpu().double().numpy()[r] - want[r]["lse"]).max() <= LSE_ATOL


def test_decoder_layers_against_the_oracle(se):
    # OmniKVDecoder over three layers (observation layer 0, sparse layers 1 and
    # 2 reading its selection): each layer's outputs against the oracle's
    # filter_step / sparse_step with the selection of layer 0
    hkv, G, d, budget, ctx = 2, 4, 64, 40, [300, 150]
    nreq = len(ctx)
    lengths = [L for L in ctx for _ in range(hkv)]
    max_pages = -(-(max(ctx) + 1) // 16) + 1
    layers = [isolated_units(lengths, max_pages, d, 60 + l, num_kv_heads=hkv, position_mode="contiguous")
              for l in range(3)]
    ins = [_inputs(nreq, hkv, G, d, 70 + 10 * l) for l in range(3)]
    npos = torch.tensor(ctx, dtype=torch.int32)
    scale = float(np.float32(1 / np.sqrt(d)))
    want = [[None] * nreq for _ in range(3)]
    for r in range(nreq):
        units = [[oracle_unit(layers[l], r * hkv + h) for h in range(hkv)] for l in range(3)]
        q, k, v = ins[0]
        f = omnikv.filter_step(units[0], f64(q[r]), f64(k[r]), f64(v[r]), ctx[r], scale, budget)
        want[0][r] = f
        for l in (1, 2):
            q, k, v = ins[l]
            want[l][r] = omnikv.sparse_step(units[l], f64(q[r]), f64(k[r]), f64(v[r]), ctx[r], scale, f["J"])
    gs = [to_device(st, DEV) for st in layers]
    views = [_view(se, g, hkv) for g in gs]
    max_len = max(ctx) + 1
    dec = se.OmniKVDecoder(G, scale, budget, [0], nreq * hkv, hkv, max_len, max_pages, d, DEV)
    for l in range(3):
        q, k, v = (t.to(DEV) for t in ins[l])
        out = torch.empty((nreq, hkv * G, d), dtype=torch.float32, device=DEV)
        lse = torch.empty((nreq, hkv * G), dtype=torch.float32, device=DEV)
        print(f"decoder layer {l}", flush=True)
        dec.layer(l, views[l], q, k, v, npos.to(DEV), out, lse, max_len)
        torch.cuda.synchronize()
        assert se.se_read_device_errors(dec.dev_err) == 0
        if l == 0:
            sel = dec.sel.cpu().numpy()
            for r in range(nreq):
                s = want[0][r]["s"]
                assert _near_tie_sets(s, sel[r].tolist(), want[0][r]["J"].tolist()), f"request {r} selection"
                if set(sel[r].tolist()) != set(want[0][r]["J"].tolist()):
                    return  # a near-tie swap: the sparse layers legitimately read other rows
        for r in range(nreq):
            np.testing.assert_allclose(out[r].cpu().numpy(), want[l][r]["o"], atol=OUT_ATOL, rtol=0)
            np.testing.assert_allclose(lse[r].cpu().numpy(), want[l][r]["lse"], atol=LSE_ATOL, rtol=0)
