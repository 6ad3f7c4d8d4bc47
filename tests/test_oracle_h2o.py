"""Pins for oracle.h2o (CPU only)."""
import json
import math
import os

import numpy as np
import pytest

from oracle import brute, h2o
from oracle.attention import selected_attention
from oracle.state import new_unit

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _unit(rng, L, d, page_size=16):
    return new_unit(rng.standard_normal((L, d)), rng.standard_normal((L, d)),
                    np.arange(L), page_size=page_size)


def test_golden_budget4_window2():
    g = json.load(open(os.path.join(GOLDEN, "h2o_budget4_window2.json")))
    B, w = g["budget"], g["recent"]
    for step in ("step1", "step2"):
        s = g[step]
        pos, u = np.array(s["pos"]), np.array(s["u"], dtype=np.float64)
        keep = h2o.retain(pos, u, B, w)
        assert sorted(pos[keep].tolist()) == s["expect_retained_pos"]
        L = len(pos)
        st = new_unit(np.arange(L, dtype=np.float64)[:, None] * np.ones((1, 2)),
                      np.zeros((L, 2)), pos, u)
        h2o.compact(st, keep, B)
        assert st.pos.tolist() == s["expect_layout_pos"]
        # keys travel with their slot (key row i was filled with the value i)
        assert st.K[:, 0].tolist() == [float(pos.tolist().index(p)) for p in s["expect_layout_pos"]]
    t = g["tie"]
    pos, u = np.array(t["pos"]), np.array(t["u"])
    assert sorted(pos[h2o.retain(pos, u, 3, 1)].tolist()) == t["budget3_window1_expect_retained_pos"]
    assert sorted(pos[h2o.retain(pos, u, 2, 1)].tolist()) == t["budget2_window1_expect_retained_pos"]


@pytest.mark.parametrize("seed", range(40))
def test_retain_matches_bruteforce_with_ties(seed):
    rng = np.random.default_rng(seed)
    L = int(rng.integers(1, 60))
    B = int(rng.integers(1, 50))
    w = int(rng.integers(0, 70))
    pos = rng.permutation(200)[:L]
    # coarse grid so that many scores tie exactly
    u = rng.integers(0, 5, size=L).astype(np.float64) / 4.0
    keep = h2o.retain(pos, u, B, w)
    expect = brute.h2o_retained_positions(pos.tolist(), u.tolist(), B, w)
    assert sorted(pos[keep].tolist()) == expect
    assert keep.sum() == min(B, L)
    if L > B:
        W = h2o.window_mask(pos, B, w)
        assert np.all(keep[W]), "the recent window is always retained"
        assert W.sum() == min(w, B)
        # the newest token is always in the window when w >= 1
        if min(w, B) >= 1:
            assert keep[np.argmax(pos)]


def test_budget_at_least_length_is_identity_and_dense():
    # TopK returns every candidate when there are fewer than b (Table
    # background-notation), so B >= L keeps everything and the step is dense attention.
    rng = np.random.default_rng(5)
    d, L, G = 8, 20, 4
    st = _unit(rng, L, d)
    before = st.copy()
    q = rng.standard_normal((G, d))
    k, v = rng.standard_normal(d), rng.standard_normal(d)
    res = h2o.decode_step(st, q, k, v, 1000, 1 / math.sqrt(d), budget=64, recent=8)
    assert st.length == L + 1
    np.testing.assert_array_equal(st.K[:L], before.K)
    keys = np.vstack([before.K, k[None]]).tolist()
    vals = np.vstack([before.V, v[None]]).tolist()
    for a in range(G):
        ob, wb, lb = brute.dense_attention(list(q[a]), keys, vals, 1 / math.sqrt(d))
        np.testing.assert_allclose(res["o"][a], ob, atol=1e-12)
        assert abs(res["lse"][a] - lb) < 1e-12
    assert res["freed"].size == 0


def test_accumulate_invariants():
    rng = np.random.default_rng(9)
    d, L, G = 8, 50, 4
    st = _unit(rng, L, d)
    st.u = rng.random(L)
    u0 = st.u.copy()
    q = rng.standard_normal((G, d))
    res = h2o.decode_step(st, q, rng.standard_normal(d), rng.standard_normal(d), 77, 0.3,
                          budget=1000, recent=4)
    u1 = res["u_after_accumulate"]
    # each head's weights sum to 1, so a KV head's scores grow by G in total
    assert abs((u1.sum() - u0.sum()) - G) < 1e-12
    # retained scores never decrease; the new token starts at 0 and ends with
    # its own summed weight
    assert np.all(u1[:L] >= u0)
    assert abs(u1[L] - res["alpha"][:, L].sum()) < 1e-15
    assert np.all(u1 >= 0)


def test_new_token_weight_from_bruteforce():
    # The new token's score after its first step equals the sum over the
    # group of its dense-attention weight (eq. background-h2o-score).
    rng = np.random.default_rng(21)
    d, L, G = 4, 6, 2
    st = _unit(rng, L, d)
    q = rng.standard_normal((G, d))
    k, v = rng.standard_normal(d), rng.standard_normal(d)
    keys = np.vstack([st.K, k[None]]).tolist()
    vals = np.vstack([st.V, v[None]]).tolist()
    res = h2o.decode_step(st, q, k, v, 99, 0.5, budget=100, recent=2)
    expect = sum(brute.dense_attention(list(q[a]), keys, vals, 0.5)[1][L] for a in range(G))
    assert abs(res["u_after_accumulate"][L] - expect) < 1e-14


@pytest.mark.parametrize("seed", range(12))
def test_compaction_properties(seed):
    # Layout parity is a convention of this repository (hole-fill); the
    # paper fixes only the retained set.  The properties below pin that the
    # oracle implements the stated convention.
    rng = np.random.default_rng(100 + seed)
    d = 4
    L = int(rng.integers(2, 80))
    B = int(rng.integers(1, L))
    w = int(rng.integers(0, B + 3))
    st = new_unit(rng.standard_normal((L, d)), rng.standard_normal((L, d)),
                  rng.permutation(500)[:L], rng.integers(0, 6, L) / 3.0)
    before = st.copy()
    keep = h2o.retain(st.pos, st.u, B, w)
    holes, movers, freed = h2o.compact(st, keep, B)
    assert st.length == B
    # slots [0, B) hold exactly the retained set, each with its own K, V, u
    assert sorted(st.pos.tolist()) == sorted(before.pos[keep].tolist())
    src = {int(p): i for i, p in enumerate(before.pos)}
    for i, p in enumerate(st.pos):
        j = src[int(p)]
        np.testing.assert_array_equal(st.K[i], before.K[j])
        np.testing.assert_array_equal(st.V[i], before.V[j])
        assert st.u[i] == before.u[j]
    # retained slots below B do not move; only the evicted count moves
    for i in range(B):
        if keep[i]:
            assert st.pos[i] == before.pos[i]
    assert len(movers) == int((~keep[:B]).sum())
    # ascending mover k lands in ascending hole k
    assert list(holes) == sorted(holes) and list(movers) == sorted(movers)
    for h, m in zip(holes, movers):
        assert st.pos[h] == before.pos[m]
    # freed logical pages: ceil(B/16) .. ceil(L/16) - 1
    assert freed.tolist() == list(range(math.ceil(B / 16), math.ceil(L / 16)))


def test_recent_token_leaving_window_competes():
    # Appendix A.3: a recent token that leaves the window must compete on its score.
    pos = np.array([0, 1, 2, 3, 4])
    u = np.array([5.0, 4.0, 3.0, 0.01, 0.5])
    # window 1 -> {4}; position 3 just left the window and has the lowest score
    keep = h2o.retain(pos, u, 4, 1)
    assert not keep[3] and keep.sum() == 4


def test_eviction_removes_entries_for_later_queries():
    # Appendix A.1: retaining only part of the cache prevents later queries
    # from reading the evicted entries; the next step reads exactly B+1 slots.
    rng = np.random.default_rng(4)
    d = 4
    st = _unit(rng, 8, d)
    q = rng.standard_normal((1, d))
    h2o.decode_step(st, q, rng.standard_normal(d), rng.standard_normal(d), 8, 1.0, budget=3, recent=1)
    assert st.length == 3
    res = h2o.decode_step(st, q, rng.standard_normal(d), rng.standard_normal(d), 9, 1.0, budget=3, recent=1)
    assert res["alpha"].shape[1] == 4
