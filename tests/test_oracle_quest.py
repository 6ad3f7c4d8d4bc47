"""Pins for oracle.quest (CPU only)."""
import json
import math
import os

import numpy as np
import pytest

from oracle import brute, quest
from oracle.state import new_unit

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_golden_strict_and_single_page_bound():
    g = json.load(open(os.path.join(GOLDEN, "quest_bound_strict.json")))
    for case in ("strict", "single"):
        c = g[case]
        keys = np.array(c["keys"])
        mn, mx = quest.page_summaries(keys, len(keys), page_size=len(keys))
        bound = quest.page_bounds(np.array([c["q"]]), mn, mx, g["scale"])[0, 0]
        assert bound == c["expect_bound"]
        assert max(float(np.dot(c["q"], k)) for k in keys) == c["expect_max_logit"]
        assert brute.quest_page_bound(c["q"], c["keys"], g["scale"]) == c["expect_bound"]


def test_golden_eight_token_example():
    g = json.load(open(os.path.join(GOLDEN, "quest_eight_tokens.json")))
    ps = g["page_size"]
    K = np.array([[x, 0.0] for x in g["history_keys_ch0"]])
    st = new_unit(K, np.arange(16, dtype=np.float64).reshape(8, 2), np.arange(8), page_size=ps)
    quest.attach_summaries(st)
    res = quest.decode_step(st, np.array([g["q"]]), np.array(g["new_key"]), np.zeros(2), 8,
                            g["scale"], g["top_k"])
    np.testing.assert_allclose(res["scores"], g["expect_scores"], atol=1e-15)
    assert res["selected"].tolist() == g["expect_selected"]
    assert res["S"].tolist() == g["expect_read_slots"]
    assert st.length == g["expect_resident"]


@pytest.mark.parametrize("seed", range(8))
def test_bound_upper_bounds_every_logit(seed):
    rng = np.random.default_rng(seed)
    d, ps, L, G = 16, 16, int(rng.integers(16, 200)), 4
    K = rng.standard_normal((L, d))
    q = rng.standard_normal((G, d))
    mn, mx = quest.page_summaries(K, L, ps)
    zhat = quest.page_bounds(q, mn, mx, 0.25)
    z = (q @ K.T) * 0.25
    for b in range(mn.shape[0]):
        rows = slice(b * ps, min((b + 1) * ps, L))
        assert np.all(zhat[:, b] >= z[:, rows].max(axis=1) - 1e-12)
        for a in range(G):
            assert abs(zhat[a, b] - brute.quest_page_bound(list(q[a]), K[rows].tolist(), 0.25)) < 1e-12


def test_single_token_pages_bound_is_exact():
    rng = np.random.default_rng(2)
    K = rng.standard_normal((10, 8))
    q = rng.standard_normal((3, 8))
    mn, mx = quest.page_summaries(K, 10, 1)
    np.testing.assert_allclose(quest.page_bounds(q, mn, mx, 0.7), (q @ K.T) * 0.7, atol=1e-13)


def test_summaries_follow_appends():
    rng = np.random.default_rng(8)
    d, ps = 8, 16
    K = rng.standard_normal((37, d))
    st = new_unit(K[:20], K[:20], np.arange(20), page_size=ps)
    quest.attach_summaries(st)
    for j in range(20, 37):
        quest.append(st, K[j], K[j], j)
    mn, mx = quest.page_summaries(K, 37, ps)
    np.testing.assert_array_equal(st.mn, mn)
    np.testing.assert_array_equal(st.mx, mx)


@pytest.mark.parametrize("seed", range(20))
def test_select_matches_bruteforce_with_ties(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(0, 80))
    top_k = int(rng.integers(1, 90))
    scores = rng.integers(-3, 3, size=n).astype(np.float64)
    sel = quest.select_pages(scores, n, top_k)
    assert sel.tolist() == brute.topk_indices(scores.tolist(), list(range(n)), top_k)
    assert len(sel) == min(top_k, n)


def test_select_all_pages_is_dense_attention():
    # Selecting every candidate page reads the whole history: dense attention.
    rng = np.random.default_rng(12)
    d, ps, L, G = 8, 16, 70, 4
    K, V = rng.standard_normal((L, d)), rng.standard_normal((L, d))
    st = new_unit(K, V, np.arange(L), page_size=ps)
    quest.attach_summaries(st)
    q = rng.standard_normal((G, d))
    k, v = rng.standard_normal(d), rng.standard_normal(d)
    res = quest.decode_step(st, q, k, v, L, 1 / math.sqrt(d), top_k=64)
    assert res["S"].tolist() == list(range(L + 1))
    keys = np.vstack([K, k[None]]).tolist()
    vals = np.vstack([V, v[None]]).tolist()
    for a in range(G):
        ob, _, lb = brute.dense_attention(list(q[a]), keys, vals, 1 / math.sqrt(d))
        np.testing.assert_allclose(res["o"][a], ob, atol=1e-12)
        assert abs(res["lse"][a] - lb) < 1e-12


def test_selection_reads_subset_and_keeps_everything():
    # Section 3.1 / Appendix A.1: selection leaves every entry resident and
    # attention over it equals dense attention over the read slots.
    rng = np.random.default_rng(13)
    d, ps, L = 8, 4, 64
    K, V = rng.standard_normal((L, d)), rng.standard_normal((L, d))
    st = new_unit(K, V, np.arange(L), page_size=ps)
    quest.attach_summaries(st)
    q = rng.standard_normal((2, d))
    res = quest.decode_step(st, q, rng.standard_normal(d), rng.standard_normal(d), L, 0.35, top_k=3)
    assert st.length == L + 1
    assert len(res["selected"]) == 3 and res["n_candidates"] == L // ps
    S = res["S"]
    assert len(S) == 3 * ps + 1
    for a in range(2):
        ob, _, _ = brute.dense_attention(list(q[a]), st.K[S].tolist(), st.V[S].tolist(), 0.35)
        np.testing.assert_allclose(res["o"][a], ob, atol=1e-12)
    # the group score is the maximum over the group's heads
    cur = (st.length - 1) // ps
    per_head = quest.page_bounds(q, st.mn[:cur], st.mx[:cur], 0.35)
    np.testing.assert_array_equal(res["scores"], per_head.max(axis=0))
