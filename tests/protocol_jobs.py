"""The oracle side of the step protocol, one unit per job (test
infrastructure; runs in the CPU workers of tests/oracle_pool.py, NumPy only).

A job gets the GPU's pre-step state of one unit (bf16 bit patterns, positions,
fp32 scores or Quest summaries) and the GPU's results of the step, runs the
oracle's step from that state and raises AssertionError on any difference
beyond the parity bars.  What needs the GPU's pools (bit-exact comparison of
the compacted key and value rows) is returned to the caller.
"""

import numpy as np

from oracle import h2o, quest
from oracle.attention import selected_attention
from oracle.state import new_unit
from tests.oracle_bridge import (H2O_NEAR_TIE, LSE_ATOL, OUT_ATOL, QUEST_RTOL, assert_scores_close, h2o_near_tie,
                                 quest_near_tie)


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (int16/uint16) -> float64, exactly."""
    b = np.asarray(bits).view(np.uint16).astype(np.uint32) << 16
    return b.view(np.float32).astype(np.float64)


def h2o_unit_job(job):
    """One H2O step of one unit.  job: where, kbits, vbits [L, d] (pre-step),
    pos [L], u fp32 [L], q float64 [G, d], k_new, v_new bits [d], p, scale,
    budget, recent, o [G, d] and lse [G] of the GPU, and acc_pos / acc_u: the
    positions and fp32 scores after the unfused call's append and update.
    Returns (holes, movers, freed, expected positions, expected fp32 scores,
    near) where near is 1 when the float64 retention differs by a near tie."""
    where = job["where"]
    st = new_unit(bf16_bits_to_f64(job["kbits"]), bf16_bits_to_f64(job["vbits"]), job["pos"],
                  job["u"].astype(np.float64))
    L1 = st.length + 1
    res = h2o.decode_step(st, job["q"], bf16_bits_to_f64(job["k_new"]), bf16_bits_to_f64(job["v_new"]),
                          int(job["p"]), job["scale"], job["budget"], job["recent"], evict=False)
    err = np.abs(job["o"] - res["o"]).max()
    assert err <= OUT_ATOL, f"{where}: output off by {err:.3e}"
    err = np.abs(job["lse"] - res["lse"]).max()
    assert err <= LSE_ATOL, f"{where}: lse off by {err:.3e}"
    # the append and the score update of the unfused call
    assert job["acc_pos"].shape[0] == L1, f"{where}: length after the append"
    assert np.array_equal(job["acc_pos"], res["pos_after_append"]), f"{where}: positions after the append"
    assert_scores_close(job["acc_u"], res["u_after_accumulate"], where)
    # retention and compaction on the GPU's own fp32 scores (the rows move with
    # their slots; the caller applies holes/movers to the key and value bits)
    u32 = job["acc_u"].astype(np.float64)
    keep = h2o.retain(res["pos_after_append"], u32, job["budget"], job["recent"])
    rows = np.zeros((L1, 0))
    st2 = new_unit(rows, rows, job["acc_pos"], u32)
    holes, movers, freed = h2o.compact(st2, keep, job["budget"])
    # the oracle's float64 selection: the same set, or a swap of near-tied scores
    near = 0
    keep64 = h2o.retain(res["pos_after_append"], res["u_after_accumulate"], job["budget"], job["recent"])
    if not np.array_equal(keep64, keep):
        p = res["pos_after_append"]
        ou = dict(zip(p.tolist(), res["u_after_accumulate"].tolist()))
        assert h2o_near_tie(ou, set(p[keep].tolist()), set(p[keep64].tolist()), H2O_NEAR_TIE), \
            f"{where}: float64 retention differs beyond a near tie"
        near = 1
    return holes, movers, freed, st2.pos, st2.u.astype(np.float32), near


def quest_summary_job(job):
    """The oracle's page summaries of one unit's resident keys must equal the
    GPU's (eq. background-quest-summary; bf16 extrema are exact)."""
    K = bf16_bits_to_f64(job["kbits"])
    mn, mx = quest.page_summaries(K, K.shape[0], 16)
    assert np.array_equal(bf16_bits_to_f64(job["meta"][:, 0]), mn), f"{job['where']}: page minima"
    assert np.array_equal(bf16_bits_to_f64(job["meta"][:, 1]), mx), f"{job['where']}: page maxima"
    return 0


def quest_unit_job(job):
    """One Quest step of one unit from the GPU's pre-step summaries.  job:
    where, q float64 [G, d], meta bits [n_cand, 2, d] (summaries of the
    candidate pages), scores fp32 [n_cand] and sel (the GPU's page scores and
    its selection), L (slots after the append), top_k, scale, kbits/vbits of
    the read set (the selected pages' rows then the current page's, as
    quest.read_set lists them), o [G, d], lse [G]; cur_k / cur_meta: the
    current page's resident key rows before the append and its summary after
    it (GPU), k_new / v_new bits.  Returns 1 when the float64 selection
    differs by a near tie."""
    where = job["where"]
    q = job["q"]
    n = job["meta"].shape[0]
    top_k = int(job["top_k"])
    mn = bf16_bits_to_f64(job["meta"][:, 0])
    mx = bf16_bits_to_f64(job["meta"][:, 1])
    want = quest.group_page_scores(q, mn, mx, job["scale"])
    s32 = job["scores"].astype(np.float64)
    if n:
        e = np.abs(s32 - want) / np.maximum(1.0, np.abs(want))
        assert e.max() <= QUEST_RTOL, f"{where}: page score off by {e.max():.3e}"
    chosen = quest.select_pages(s32, n, top_k)
    kk = min(top_k, n)
    assert np.array_equal(job["sel"][:kk], chosen), f"{where}: selection differs on the GPU's scores"
    assert (job["sel"][kk:] == -1).all(), f"{where}: selection padding"
    near = 0
    sel64 = quest.select_pages(want, n, top_k)
    if not np.array_equal(sel64, chosen):
        assert quest_near_tie(want, chosen, sel64), f"{where}: float64 selection differs beyond a near tie"
        near = 1
    S = quest.read_set(chosen, int(job["L"]), 16)
    assert S.shape[0] == job["kbits"].shape[0], f"{where}: read set size"
    K = bf16_bits_to_f64(job["kbits"])
    V = bf16_bits_to_f64(job["vbits"])
    o, lse, _, _ = selected_attention(q, K, V, np.arange(S.shape[0]), job["scale"])
    err = np.abs(job["o"] - o).max()
    assert err <= OUT_ATOL, f"{where}: output off by {err:.3e}"
    assert np.abs(job["lse"] - lse).max() <= LSE_ATOL, f"{where}: lse"
    # the append folds the new key into the current page's summary
    cur = bf16_bits_to_f64(job["cur_k"])
    st = new_unit(cur, cur, np.arange(cur.shape[0]))
    quest.attach_summaries(st)
    quest.append(st, bf16_bits_to_f64(job["k_new"]), bf16_bits_to_f64(job["v_new"]), 0)
    assert np.array_equal(bf16_bits_to_f64(job["cur_meta"][0]), st.mn[-1]), f"{where}: page minimum after append"
    assert np.array_equal(bf16_bits_to_f64(job["cur_meta"][1]), st.mx[-1]), f"{where}: page maximum after append"
    return near
