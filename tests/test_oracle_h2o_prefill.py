"""Pins of the oracle's H2O chunk-wise prefill eviction (oracle/h2o.py
prefill_chunk): a hand-derived two-chunk-token fixture, brute-force scores and
retention in pure Python, the single-token case against the decode recurrence,
and invariants."""
import json
import os

import numpy as np
import pytest

from oracle import brute, h2o
from oracle.state import new_unit

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_golden_chunk():
    g = json.load(open(os.path.join(GOLDEN, "h2o_prefill_chunk.json")))
    r = g["resident"]
    st = new_unit(np.array(r["K"]), np.array(r["K"]), np.array(r["pos"]), np.array(r["u"]))
    c = g["chunk"]
    res = h2o.prefill_chunk(st, np.array(c["K"]), np.array(c["K"]), np.array(c["pos"]), np.array(g["Qs"]),
                            g["scale"], g["budget"], g["recent"])
    np.testing.assert_allclose(res["u_after_accumulate"], g["expect_u_after_accumulate"], rtol=0, atol=1e-15)
    np.testing.assert_array_equal(st.pos, g["expect_pos"])
    np.testing.assert_allclose(st.u, g["expect_u"], rtol=0, atol=1e-15)


@pytest.mark.parametrize("L0,C,s,G,B,w", [(0, 12, 12, 1, 8, 3), (10, 9, 4, 2, 12, 5), (7, 6, 1, 4, 20, 4)])
def test_brute_force_scores_and_retention(L0, C, s, G, B, w):
    rng = np.random.default_rng(L0 * 31 + C)
    d, scale = 6, 0.4
    pos0 = rng.permutation(3 * L0 + 1)[:L0]           # resident positions in any slot order
    K0, V0 = rng.standard_normal((L0, d)), rng.standard_normal((L0, d))
    u0 = rng.random(L0)
    base = int(pos0.max()) + 1 if L0 else 0
    pos_c = base + np.arange(C) * 2                    # increasing, above the resident ones
    Kc, Vc = rng.standard_normal((C, d)), rng.standard_normal((C, d))
    Qs = rng.standard_normal((s, G, d))
    st = new_unit(K0, V0, pos0, u0)
    res = h2o.prefill_chunk(st, Kc, Vc, pos_c, Qs, scale, B, w)
    # brute force: every scoring query over the slots up to its position
    Kall = [list(r) for r in np.vstack([K0, Kc])] if L0 else [list(r) for r in Kc]
    Pall = list(pos0) + list(pos_c)
    u = list(u0) + [0.0] * C
    for t in range(s):
        p_t = pos_c[C - s + t]
        vis = [j for j in range(L0 + C) if Pall[j] <= p_t]
        for a in range(G):
            _, wts, _ = brute.dense_attention(list(Qs[t, a]), [Kall[j] for j in vis], [Kall[j] for j in vis], scale)
            for j, x in zip(vis, wts):
                u[j] += x
    np.testing.assert_allclose(res["u_after_accumulate"], u, rtol=0, atol=1e-12)
    want = brute.h2o_retained_positions(Pall, u, B, w)
    assert sorted(st.pos.tolist()) == want
    assert abs(sum(u) - sum(u0) - s * G) < 1e-9        # every query head's weights sum to 1


def test_single_token_chunk_is_the_decode_recurrence():
    rng = np.random.default_rng(3)
    L0, d, G, B, w, scale = 30, 8, 4, 20, 6, 0.3
    K0, V0 = rng.standard_normal((L0, d)), rng.standard_normal((L0, d))
    pos0, u0 = np.arange(L0), rng.random(L0)
    k, v, q = rng.standard_normal(d), rng.standard_normal(d), rng.standard_normal((G, d))
    a, b = new_unit(K0, V0, pos0, u0), new_unit(K0, V0, pos0, u0)
    h2o.decode_step(a, q, k, v, L0, scale, B, w)
    h2o.prefill_chunk(b, k[None], v[None], np.array([L0]), q[None], scale, B, w)
    np.testing.assert_array_equal(a.pos, b.pos)
    np.testing.assert_allclose(a.u, b.u, rtol=0, atol=1e-14)
    np.testing.assert_array_equal(a.K, b.K)


def test_budget_covering_everything_keeps_all():
    rng = np.random.default_rng(4)
    st = new_unit(rng.standard_normal((5, 4)), rng.standard_normal((5, 4)), np.arange(5))
    res = h2o.prefill_chunk(st, rng.standard_normal((3, 4)), rng.standard_normal((3, 4)), np.arange(5, 8),
                            rng.standard_normal((2, 2, 4)), 0.5, 8, 2)
    assert st.length == 8 and res["keep"].all()
