"""Pins of the SnapKV oracle (oracle/snapkv.py) to the paper and to
mathematics that is not the oracle's own code: hand-derived fixtures, a
closed form, invariants and a constructed case with a known selection."""
import json
import os

import numpy as np
import pytest

from oracle import snapkv
from oracle.state import new_unit

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def test_golden_three_keys():
    g = _load("snapkv_three_keys.json")
    K, pos = np.array(g["K"]), np.array(g["pos"])
    for key, w in (("w1", 1), ("w2", 2)):
        u = snapkv.observation_scores(np.array(g[key]["Qo"]), K, pos, w, g["scale"])
        for j, want in g[key]["expect_u_candidates"].items():
            assert u[int(j)] == pytest.approx(want, abs=1e-15)


@pytest.mark.parametrize("kappa", [1, 3, 5])
def test_golden_pool_max(kappa):
    g = _load("snapkv_pool_max.json")
    pos, u = np.array(g["pos"]), np.array(g["u"])
    cand = np.ones(len(pos), dtype=bool)
    cand[g["window"]] = False
    s = snapkv.pool_max(u, pos, cand, kappa)
    np.testing.assert_array_equal(s[cand], np.array(g["expect"][str(kappa)]))
    assert (s[~cand] == 0).all()


@pytest.mark.parametrize("L,w,G", [(37, 5, 1), (64, 8, 4), (130, 3, 2)])
def test_zero_queries_closed_form(L, w, G):
    # q = 0: every logit is 0, so query t (at position L-w+t) spreads weight
    # 1/(L-w+t+1) over the keys at positions <= its own; a candidate collects
    # G * sum_t 1/(L-w+t+1).
    rng = np.random.default_rng(L)
    K = rng.standard_normal((L, 16))
    u = snapkv.observation_scores(np.zeros((w, G, 16)), K, np.arange(L), w, 0.125)
    want = G * sum(1.0 / (L - w + t + 1) for t in range(w))
    np.testing.assert_allclose(u[:L - w], want, rtol=0, atol=1e-13)


def test_total_weight_is_w_times_g():
    # every (observation query, query head) softmax sums to 1 over what it reads
    rng = np.random.default_rng(3)
    L, w, G = 90, 7, 4
    u = snapkv.observation_scores(rng.standard_normal((w, G, 32)), rng.standard_normal((L, 32)),
                                  np.arange(L) * 3 + 5, w, 0.2)
    assert u.sum() == pytest.approx(w * G, abs=1e-12)
    assert (u >= 0).all()


def test_positions_not_slots_define_causality_and_window():
    # shuffling the slots (with their positions) permutes u and s the same way
    rng = np.random.default_rng(7)
    L, w, G, d = 50, 6, 2, 8
    K, Qo = rng.standard_normal((L, d)), rng.standard_normal((w, G, d))
    pos = np.arange(L)
    perm = rng.permutation(L)
    u1 = snapkv.observation_scores(Qo, K, pos, w, 0.4)
    u2 = snapkv.observation_scores(Qo, K[perm], pos[perm], w, 0.4)
    np.testing.assert_allclose(u2, u1[perm], rtol=1e-13, atol=1e-15)
    cand = pos < L - w
    s1 = snapkv.pool_max(u1, pos, cand, 7)
    s2 = snapkv.pool_max(u2, pos[perm], cand[perm], 7)
    np.testing.assert_allclose(s2, s1[perm], rtol=1e-13, atol=1e-15)


def test_eight_token_prompt_pooling_promotes_neighbours():
    # The paper's eight-token shape (w = 2, B = 4: the last two positions plus
    # two earlier ones).  Keys k_j = (x_j, 0) and queries (8, 0): the weight
    # concentrates on x = 5 (position 5), then x = 3 (position 2).  Without
    # pooling the two earlier picks are 5 and 2; with kappa = 3, position 4
    # shares position 5's pooled score (its neighbourhood reaches 5), the tie
    # goes to the lower position, so 4 and 5 are kept and 2 is not.
    x = np.array([0.0, 0.0, 3.0, 0.0, 0.0, 5.0, 0.0, 0.0])
    K = np.stack([x, np.zeros(8)], axis=1)
    Qo = np.array([[[8.0, 0.0]], [[8.0, 0.0]]])
    for kappa, want in ((1, {2, 5, 6, 7}), (3, {4, 5, 6, 7})):
        st = new_unit(K, K, np.arange(8))
        r = snapkv.compact_prompt(st, Qo, 2, kappa, 4, 1.0)
        assert set(np.flatnonzero(r["keep"]).tolist()) == want, kappa
        assert sorted(st.pos.tolist()) == sorted(want)


@pytest.mark.parametrize("L,w,B,kappa", [(200, 16, 64, 7), (100, 32, 32, 7), (80, 8, 120, 3)])
def test_compaction_structure(L, w, B, kappa):
    rng = np.random.default_rng(L + B)
    d, G = 16, 4
    K, V = rng.standard_normal((L, d)), rng.standard_normal((L, d))
    st = new_unit(K, V, np.arange(L))
    r = snapkv.compact_prompt(st, rng.standard_normal((w, G, d)), w, kappa, B, 0.25)
    n_keep = min(B, L)
    assert int(r["keep"].sum()) == n_keep and st.length == n_keep
    if L <= B:                                                   # fits: left as it is
        np.testing.assert_array_equal(st.K, K)
        return
    assert set(range(L - w, L)) <= set(st.pos.tolist())          # O is retained
    kept = set(st.pos.tolist())
    for j in range(L - w):                                       # no dropped candidate beats a kept one
        if j not in kept:
            assert all((r["s"][j], -j) < (r["s"][k], -k) for k in kept if k < L - w)
    for row, p in zip(st.K, st.pos):                              # rows travel with their positions
        np.testing.assert_array_equal(row, K[p])
