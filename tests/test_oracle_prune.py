"""Pins of the oracle's interval prefix-cache pruning (oracle/prune.py): a
hand-derived fixture for both selection modes, pure-Python walks of the set
algebra and of the budget selection, and invariants (identity, zero budget,
untouched prefix outside the interval, attention over the pruned cache,
rebuilt Quest summaries)."""
import json
import os

import numpy as np
import pytest

from oracle import brute, prune, quest
from oracle.attention import selected_attention
from oracle.state import new_unit

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _fixture_unit(g):
    n = len(g["positions"])
    ids = np.arange(n, dtype=np.float64)[:, None]
    return new_unit(ids, ids, np.array(g["positions"]), np.array(g["scores"]), page_size=g["page_size"])


def test_golden_mask():
    g = json.load(open(os.path.join(GOLDEN, "prune_interval.json")))
    st = _fixture_unit(g)
    I = prune.mask_selection(st, g["lo"], g["hi"], np.array(g["mask"]))
    e = g["expect_mask"]
    np.testing.assert_array_equal(I, e["I"])
    r = prune.prune(st, g["lo"], g["hi"], I)
    np.testing.assert_array_equal(st.pos, e["positions"])
    np.testing.assert_array_equal(st.K[:, 0], e["old_slots"])      # rows travel with their positions
    np.testing.assert_array_equal(st.u, np.array(g["scores"])[e["old_slots"]])
    np.testing.assert_array_equal(r["freed"], e["freed"])


@pytest.mark.parametrize("case", range(4))
def test_golden_budget(case):
    g = json.load(open(os.path.join(GOLDEN, "prune_interval.json")))
    e = g["expect_budget"][case]
    st = _fixture_unit(g)
    I = prune.budget_selection(st, g["lo"], g["hi"], e["budget"])
    np.testing.assert_array_equal(I, e["I"])
    r = prune.prune(st, g["lo"], g["hi"], I)
    np.testing.assert_array_equal(st.pos, e["positions"])
    np.testing.assert_array_equal(r["freed"], e["freed"])


def _random_unit(rng, L, d=3, page_size=4, span=None):
    span = span or 3 * L + 2
    pos = rng.permutation(span)[:L]                     # resident positions in any slot order
    u = np.round(rng.random(L) * 4) / 4                  # coarse scores: ties happen
    return new_unit(rng.standard_normal((L, d)), rng.standard_normal((L, d)), pos, u, page_size=page_size)


@pytest.mark.parametrize("seed", range(12))
def test_walk_of_the_set_algebra(seed):
    rng = np.random.default_rng(seed)
    L = int(rng.integers(0, 40))
    st = _random_unit(rng, L)
    span = 3 * L + 2
    lo = int(rng.integers(-2, span + 2))
    hi = int(rng.integers(lo - 1, span + 4))
    positions = st.pos.tolist()
    if seed % 2:
        mask = rng.integers(0, 2, max(hi - lo, 0))
        I = prune.mask_selection(st, lo, hi, mask)
        want_I = {p for p in positions if lo <= p < hi and mask[p - lo]}
    else:
        b = int(rng.integers(0, 12))
        I = prune.budget_selection(st, lo, hi, b)
        want_I = brute.interval_budget_keep(positions, st.u.tolist(), lo, hi, b)
    assert set(I.tolist()) == want_I
    before = st.copy()
    r = prune.prune(st, lo, hi, I)
    stay = brute.pruned_slots(positions, lo, hi, want_I)
    assert st.pos.tolist() == [positions[s] for s in stay]
    np.testing.assert_array_equal(st.K, before.K[stay])
    np.testing.assert_array_equal(st.V, before.V[stay])
    np.testing.assert_array_equal(st.u, before.u[stay])
    np.testing.assert_array_equal(r["dest"], np.arange(len(stay)))
    assert r["freed"].tolist() == list(range(-(-len(stay) // 4), -(-L // 4)))


def test_identity_zero_budget_and_untouched_prefix():
    rng = np.random.default_rng(7)
    st = _random_unit(rng, 60, page_size=16, span=200)
    lo, hi = 40, 120
    inside = prune.in_interval(st.pos, lo, hi)
    # I = R intersected with T: nothing changes
    s1 = st.copy()
    prune.prune(s1, lo, hi, st.pos[inside])
    np.testing.assert_array_equal(s1.pos, st.pos)
    np.testing.assert_array_equal(s1.K, st.K)
    # zero budget: no position of the interval survives, every other one does, in order
    s2 = st.copy()
    r = prune.prune(s2, lo, hi, prune.budget_selection(s2, lo, hi, 0))
    assert not prune.in_interval(s2.pos, lo, hi).any()
    np.testing.assert_array_equal(s2.pos, st.pos[~inside])
    assert r["freed"].tolist() == list(range(-(-s2.length // 16), -(-st.length // 16)))
    # an interval holding no resident position leaves the unit unchanged
    s3 = st.copy()
    prune.prune(s3, 1000, 2000, [])
    np.testing.assert_array_equal(s3.pos, st.pos)
    with pytest.raises(ValueError):
        prune.retained_positions(st.pos.tolist(), lo, hi, [int(st.pos[~inside][0])])


def test_attention_over_the_pruned_cache():
    # attention after pruning reads exactly R': it equals brute-force dense
    # attention over the original rows whose positions stay
    rng = np.random.default_rng(3)
    st = _random_unit(rng, 30, d=4, span=50)
    q = rng.standard_normal((2, 4))
    lo, hi = 10, 35
    I = prune.budget_selection(st, lo, hi, 5)
    keep_pos = prune.retained_positions(st.pos.tolist(), lo, hi, I)
    rows = [s for s in range(st.length) if int(st.pos[s]) in keep_pos]
    before = st.copy()
    prune.prune(st, lo, hi, I)
    o, lse, _, _ = selected_attention(q, st.K, st.V, np.arange(st.length), 0.5)
    for a in range(2):
        ob, _, lb = brute.dense_attention(q[a].tolist(), before.K[rows].tolist(), before.V[rows].tolist(), 0.5)
        np.testing.assert_allclose(o[a], ob, rtol=1e-12, atol=1e-12)
        assert abs(lse[a] - lb) < 1e-12


def test_quest_summaries_rebuilt():
    rng = np.random.default_rng(11)
    st = _random_unit(rng, 37, d=5, page_size=4, span=80)
    quest.attach_summaries(st)
    prune.prune(st, 20, 60, prune.budget_selection(st, 20, 60, 3))
    n_pages = -(-st.length // 4)
    assert st.mn.shape[0] == n_pages
    for b in range(n_pages):
        rows = st.K[4 * b:min(4 * b + 4, st.length)].tolist()
        for c in range(5):
            assert st.mn[b, c] == min(r[c] for r in rows)
            assert st.mx[b, c] == max(r[c] for r in rows)
