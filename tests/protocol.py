"""Step-by-step parity protocol for the decode steps (test infrastructure).

The GPU runs the same calls, with the same per-step length bounds (and so the
same launch shapes and kernel paths), that the benchmark times.  Each step,
for every checked unit:

  * the unit's pre-step state is read back from the GPU and the oracle takes
    the step from it (re-sync: a near-tie decided one way on the GPU never
    makes later steps of the oracle diverge, and no unit is ever dropped);
  * outputs and lse are compared with the oracle's (|d| <= 1e-2 / 1e-3);
  * H2O: an unfused attention call (se_decode_attend with the score update, at
    the same launch shape) runs on a copy of the layer's pre-step state; its
    fp32 scores after the update are compared with the oracle's (1e-3
    relative), and the oracle's retention and compaction fed those same fp32
    scores must equal what the fused step left behind bit for bit: positions,
    K and V bits, scores, length and freed pages.  The oracle's own float64
    selection may differ from it only between near-tied scores (checked, not
    skipped);
  * Quest: se_quest_select on the pre-step state gives the GPU's fp32 page
    scores (the same per-page arithmetic as the fused step's bound); the
    oracle's bounds from the GPU's pre-step summaries are compared with them
    (1e-3 relative), the oracle's top-k over those same fp32 scores must equal
    the fused step's selection exactly, and the output is compared with the
    oracle's attention over that selection.  The appended token's page summary
    must equal the oracle's fold of the new key, and nothing else in the pools
    may change.

The oracle's per-unit work runs in the CPU workers of tests/oracle_pool.py
(tests/protocol_jobs.py).  Nothing here computes any part of the method; it
gathers GPU state, hands it to the oracle and compares.
"""

import numpy as np
import torch

from tests import oracle_pool
from tests.protocol_jobs import h2o_unit_job, quest_summary_job, quest_unit_job
from workloads import PagedInputs, scaled

PAGE = 16


# ----------------------------------------------------------------- GPU state readers

def read_units(gs: PagedInputs, rows, lengths=None, chunk: int = 64, with_kv: bool = True):
    """Slot-ordered state of the units at block-table rows ``rows``: a list of
    dicts with K, V (int16 bf16 bit patterns [L, d], or None without with_kv),
    pos (int64 [L]) and u (float32 [L], or None).  Gathered on the device a
    chunk of units at a time."""
    rows = [int(r) for r in rows]
    if lengths is None:
        lengths = gs.lengths[torch.tensor(rows, dtype=torch.int64, device=gs.lengths.device)].cpu().tolist()
    res = []
    dev = gs.kv_pool.device
    for c0 in range(0, len(rows), chunk):
        rr = rows[c0:c0 + chunk]
        ll = [int(x) for x in lengths[c0:c0 + chunk]]
        lmax = max(max(ll), 1)
        npages = -(-lmax // PAGE)
        bt = gs.block_table[torch.tensor(rr, dtype=torch.int64, device=dev), :npages].to(torch.int64)
        s = torch.arange(lmax, device=dev)
        page = bt[:, s // PAGE]                       # [n, lmax]
        row = (s % PAGE)[None, :].expand_as(page)
        kv = gs.kv_pool[page, :, row].view(torch.int16).cpu().numpy() if with_kv else None  # [n, lmax, 2, d]
        pos = gs.pos_pool[page, row].cpu().numpy().astype(np.int64)
        u = None if gs.score_pool is None else gs.score_pool[page, row].cpu().numpy()
        for i, L in enumerate(ll):
            res.append({"K": None if kv is None else np.ascontiguousarray(kv[i, :L, 0]),
                        "V": None if kv is None else np.ascontiguousarray(kv[i, :L, 1]),
                        "pos": pos[i, :L].copy(), "u": None if u is None else u[i, :L].copy()})
    return res


def layer_clone(gs: PagedInputs, layer: int) -> PagedInputs:
    """A compact device copy of one layer's units (their pages in block-table
    order, the identity block table): calls on it see the same per-unit data,
    the same number of units and the same bounds, hence the same launch
    shapes, as calls on the layer itself."""
    rows = gs.layer_rows(layer)
    bt = gs.block_table[rows].to(torch.int64)
    U, P = bt.shape
    flat = bt.reshape(-1)

    def take(t):
        return None if t is None else t.index_select(0, flat)

    return PagedInputs(w=scaled(gs.w, layers=1), kv_pool=take(gs.kv_pool), pos_pool=take(gs.pos_pool),
                       score_pool=take(gs.score_pool), meta_pool=take(gs.meta_pool),
                       block_table=torch.arange(U * P, dtype=torch.int32, device=bt.device).view(U, P),
                       lengths=gs.lengths[rows].clone(), max_pages=P, ctx=gs.ctx, uvec=gs.uvec)


def _bits(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().contiguous().view(torch.int16).numpy()


# ----------------------------------------------------------------- H2O

def _check_compaction(pre, post, k_bits, v_bits, result, budget, freed_gpu, fcount_gpu, bt_row, where):
    """The fused step's pools after the step against the oracle's compaction
    (holes <- movers applied to the pre-step rows plus the appended one)."""
    holes, movers, freed, exp_pos, exp_u, _ = result
    kb = np.concatenate([pre["K"], k_bits[None, :]])
    vb = np.concatenate([pre["V"], v_bits[None, :]])
    kb[holes] = kb[movers]
    vb[holes] = vb[movers]
    n_keep = min(kb.shape[0], budget)
    assert post["pos"].shape[0] == n_keep, f"{where}: length after the eviction"
    assert np.array_equal(post["pos"], exp_pos), f"{where}: positions after the eviction"
    assert np.array_equal(post["K"], kb[:n_keep]), f"{where}: key rows after the eviction"
    assert np.array_equal(post["V"], vb[:n_keep]), f"{where}: value rows after the eviction"
    assert np.array_equal(post["u"].view(np.uint32), exp_u.view(np.uint32)), f"{where}: scores after the eviction"
    assert int(fcount_gpu) == len(freed), f"{where}: freed count"
    assert np.array_equal(freed_gpu[:len(freed)], bt_row[freed]), f"{where}: freed pages"


def h2o_trajectory(se, gs: PagedInputs, steps, n_steps, check, *, q_per_kv, scale, budget, recent, bounds,
                   device, log=print):
    """Runs n_steps fused H2O steps (se_decode_step_h2o, one call per layer,
    max_len = bounds[t]) on ``gs`` and checks the units ``check`` = {layer:
    [unit index within the layer]} at every step.  Returns (unit-steps
    checked, unit-steps whose float64 retention differed by a near tie)."""
    w = gs.w
    U, G, d = w.units_per_layer, q_per_kv, w.head_dim
    P = gs.max_pages
    cap = P * PAGE
    views = [se.KVView(gs.kv_pool, gs.pos_pool, gs.score_pool, gs.meta_pool, gs.block_table[gs.layer_rows(l)],
                       gs.lengths[gs.layer_rows(l)], num_kv_heads=w.hkv) for l in range(w.layers)]
    ws = torch.empty(max(1, se.se_workspace_bytes(se.SE_OP_DECODE_ATTEND, U, cap, P, G, d)), dtype=torch.uint8,
                     device=device)
    err = torch.zeros(1, dtype=torch.int32, device=device)
    freed = torch.full((U, P), -5, dtype=torch.int32, device=device)
    fcount = torch.full((U,), -5, dtype=torch.int32, device=device)
    hq = w.hkv * G
    out = torch.empty((w.num_req, hq, d), dtype=torch.float32, device=device)
    lse = torch.empty((w.num_req, hq), dtype=torch.float32, device=device)
    cout, clse = torch.empty_like(out), torch.empty_like(lse)
    check = {int(l): sorted(int(u) for u in us) for l, us in check.items() if len(us)}
    pre = {l: read_units(gs, [l * U + u for u in us]) for l, us in check.items()}
    n_checked = n_near = 0
    for t in range(n_steps):
        ml = int(bounds[t])
        log(f"step {t}: max_len {ml}", flush=True)
        for l in range(w.layers):
            q, kn, vn, npos = steps.q[t, l], steps.k_new[t, l], steps.v_new[t, l], steps.new_pos[t]
            units = check.get(l)
            if units:
                clone = layer_clone(gs, l)
                cview = se.KVView(clone.kv_pool, clone.pos_pool, clone.score_pool, None, clone.block_table,
                                  clone.lengths, num_kv_heads=w.hkv)
                se.se_decode_attend(cview, G, q, kn, vn, npos, None, 0, scale, ml, se.SE_ATTEND_ACCUMULATE, cout,
                                    clse, None, 0, ws, err)
                fcount.fill_(-5)
            se.se_decode_step_h2o(views[l], G, q, kn, vn, npos, scale, budget, recent, ml, out, lse, freed, P,
                                  fcount, ws, err)
            if not units:
                continue
            torch.cuda.synchronize()
            assert se.se_read_device_errors(err) == 0, f"step {t} layer {l}: device error"
            # the fused call's attention is the unfused call's, launch for launch
            assert torch.equal(out, cout), f"step {t} layer {l}: fused and unfused outputs differ"
            assert torch.equal(lse, clse), f"step {t} layer {l}: fused and unfused lse differ"
            acc = read_units(clone, units, with_kv=False)
            del clone, cview
            post = read_units(gs, [l * U + u for u in units])
            o_g, lse_g = out.cpu().double().numpy(), lse.cpu().double().numpy()
            fr, fc = freed.cpu().numpy(), fcount.cpu().numpy()
            bt = gs.block_table[gs.layer_rows(l)].cpu().numpy()
            qh = steps.q[t, l].cpu().to(torch.float64).numpy()
            kb, vb, ph = _bits(steps.k_new[t, l]), _bits(steps.v_new[t, l]), steps.new_pos[t].cpu().numpy()
            jobs = []
            for i, u in enumerate(units):
                req, kvh = divmod(u, w.hkv)
                rows = slice(kvh * G, (kvh + 1) * G)
                jobs.append({"where": f"step {t} layer {l} unit {u}", "kbits": pre[l][i]["K"],
                             "vbits": pre[l][i]["V"], "pos": pre[l][i]["pos"], "u": pre[l][i]["u"],
                             "q": qh[req, rows], "k_new": kb[req, kvh], "v_new": vb[req, kvh], "p": int(ph[req]),
                             "scale": scale, "budget": budget, "recent": recent, "o": o_g[req, rows],
                             "lse": lse_g[req, rows], "acc_pos": acc[i]["pos"], "acc_u": acc[i]["u"]})
            results = oracle_pool.run(h2o_unit_job, jobs)
            for i, u in enumerate(units):
                req, kvh = divmod(u, w.hkv)
                _check_compaction(pre[l][i], post[i], kb[req, kvh], vb[req, kvh], results[i], budget, fr[u], fc[u],
                                  bt[u], f"step {t} layer {l} unit {u}")
                n_near += results[i][5]
            n_checked += len(units)
            pre[l] = post
    return n_checked, n_near


# ----------------------------------------------------------------- Quest

def quest_trajectory(se, gs: PagedInputs, steps, n_steps, units, *, q_per_kv, scale, top_k, bounds, device,
                     log=print):
    """Runs n_steps fused Quest steps (se_decode_step_quest, max_len =
    bounds[t]) on a single-layer ``gs`` (summaries built by
    se_quest_summarize) and checks ``units`` at every step.  Returns (unit-steps
    checked, unit-steps whose float64 selection differed by a near tie)."""
    w = gs.w
    U, G, d = w.units_per_layer, q_per_kv, w.head_dim
    P = gs.max_pages
    cap = P * PAGE
    view = se.KVView(gs.kv_pool, gs.pos_pool, gs.score_pool, gs.meta_pool, gs.block_table, gs.lengths,
                     num_kv_heads=w.hkv)
    err = torch.zeros(1, dtype=torch.int32, device=device)
    ws = torch.empty(max(1, se.se_workspace_bytes(se.SE_OP_QUEST_STEP, U, cap, P, G, d, top_k)), dtype=torch.uint8,
                     device=device)
    ws_sel = torch.empty(max(1, se.se_workspace_bytes(se.SE_OP_QUEST_SELECT, U, cap, P, G, d)), dtype=torch.uint8,
                         device=device)
    sel = torch.full((U, top_k), -3, dtype=torch.int32, device=device)
    sel_ref = torch.full((U, top_k), -3, dtype=torch.int32, device=device)
    scores = torch.full((U, P), float("nan"), dtype=torch.float32, device=device)
    hq = w.hkv * G
    out = torch.empty((w.num_req, hq, d), dtype=torch.float32, device=device)
    lse = torch.empty((w.num_req, hq), dtype=torch.float32, device=device)
    se.se_quest_summarize(view, cap, err)
    torch.cuda.synchronize()
    assert se.se_read_device_errors(err) == 0
    units = sorted(int(u) for u in units)
    bt_all = gs.block_table.to(torch.int64)

    def meta_bits(u, n):
        return gs.meta_pool[bt_all[u, :n]].view(torch.int16).cpu().numpy()   # [n, 2, d]

    # the summaries se_quest_summarize built, against the oracle's
    log(f"checking the summaries of {len(units)} units", flush=True)
    for c0 in range(0, len(units), 64):
        part = units[c0:c0 + 64]
        st = read_units(gs, part)
        jobs = [{"where": f"unit {u}", "kbits": st[i]["K"], "meta": meta_bits(u, -(-st[i]["K"].shape[0] // PAGE))}
                for i, u in enumerate(part)]
        oracle_pool.run(quest_summary_job, jobs)
    n_checked = n_near = 0
    for t in range(n_steps):
        ml = int(bounds[t])
        log(f"step {t}: max_len {ml}", flush=True)
        q, kn, vn, npos = steps.q[t, 0], steps.k_new[t, 0], steps.v_new[t, 0], steps.new_pos[t]
        L0 = gs.lengths.cpu().numpy().astype(np.int64)
        meta0 = {u: meta_bits(u, int(L0[u]) // PAGE) for u in units}   # the candidates' summaries
        cur0 = {}
        for u in units:
            r = int(L0[u]) % PAGE
            ph_ = int(bt_all[u, int(L0[u]) // PAGE])
            cur0[u] = _bits(gs.kv_pool[ph_, 0, :r])
        kv_before, pos_before, meta_before = gs.kv_pool.clone(), gs.pos_pool.clone(), gs.meta_pool.clone()
        se.se_quest_select(view, G, q, scale, top_k, ml, 0, sel_ref, scores, P, ws_sel, err)
        se.se_decode_step_quest(view, G, q, kn, vn, npos, scale, top_k, ml, sel, out, lse, ws, err)
        torch.cuda.synchronize()
        assert se.se_read_device_errors(err) == 0, f"step {t}: device error"
        assert torch.equal(sel, sel_ref), f"step {t}: fused and two-call selections differ"
        # nothing but the appended slot and its page's summary changed
        L1 = gs.lengths.cpu().numpy().astype(np.int64)
        assert np.array_equal(L1, L0 + 1), f"step {t}: lengths after the append"
        s = torch.as_tensor(L0, device=device)
        pg = bt_all[torch.arange(U, device=device), s // PAGE]
        kv_before[pg, 0, s % PAGE] = kn.reshape(U, d)
        kv_before[pg, 1, s % PAGE] = vn.reshape(U, d)
        pos_before[pg, s % PAGE] = npos.repeat_interleave(w.hkv)
        meta_before[pg] = gs.meta_pool[pg]
        assert torch.equal(kv_before, gs.kv_pool), f"step {t}: key/value rows other than the appended ones changed"
        assert torch.equal(pos_before, gs.pos_pool), f"step {t}: positions other than the appended ones changed"
        assert torch.equal(meta_before, gs.meta_pool), f"step {t}: summaries of other pages changed"
        del kv_before, pos_before, meta_before
        sel_g, sc_g = sel.cpu().numpy(), scores.cpu().numpy()
        o_g, lse_g = out.cpu().double().numpy(), lse.cpu().double().numpy()
        qh = steps.q[t, 0].cpu().to(torch.float64).numpy()
        kb, vb = _bits(kn), _bits(vn)
        jobs = []
        for u in units:
            req, kvh = divmod(u, w.hkv)
            rows = slice(kvh * G, (kvh + 1) * G)
            n = int(L0[u]) // PAGE
            L = int(L1[u])
            kk = min(top_k, n)
            pages = list(int(b) for b in sel_g[u, :kk]) + [(L - 1) // PAGE]
            slots = [b * PAGE + r for b in pages for r in range(min(PAGE, L - b * PAGE))]
            sl = torch.tensor(slots, dtype=torch.int64, device=device)
            rows_kv = gs.kv_pool[bt_all[u, sl // PAGE], :, sl % PAGE].view(torch.int16).cpu().numpy()
            cur_page = int(bt_all[u, (L - 1) // PAGE])
            jobs.append({"where": f"step {t} unit {u}", "q": qh[req, rows], "meta": meta0[u],
                         "scores": sc_g[u, :n].copy(), "sel": sel_g[u].copy(), "L": L, "top_k": top_k, "scale": scale,
                         "kbits": np.ascontiguousarray(rows_kv[:, 0]), "vbits": np.ascontiguousarray(rows_kv[:, 1]),
                         "o": o_g[req, rows], "lse": lse_g[req, rows], "cur_k": cur0[u],
                         "cur_meta": gs.meta_pool[cur_page].view(torch.int16).cpu().numpy(),
                         "k_new": kb[req, kvh], "v_new": vb[req, kvh]})
        n_near += sum(oracle_pool.run(quest_unit_job, jobs))
        n_checked += len(units)
    return n_checked, n_near
