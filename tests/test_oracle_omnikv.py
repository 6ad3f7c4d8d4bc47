"""Pins of the OmniKV oracle (oracle/omnikv.py) to the paper and to code that
is not the oracle's own: a hand-derived fixture, the paper's reuse example
against brute-force dense attention, brute-force selection with ties, and the
budget-covers-all case."""
import json
import os

import numpy as np
import pytest

from oracle import brute, omnikv
from oracle.state import new_unit

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_golden_max_over_heads():
    g = json.load(open(os.path.join(GOLDEN, "omnikv_max_over_heads.json")))
    q = np.array(g["q"])
    K = [np.array(k) for k in g["K_heads"]]
    s = omnikv.position_scores(q, K, g["q_per_kv"], g["scale"])
    np.testing.assert_allclose(s, g["expect_s"], rtol=0, atol=1e-15)
    for b, want in g["expect_J"].items():
        np.testing.assert_array_equal(omnikv.select(s, int(b)), want)


@pytest.mark.parametrize("L,b,levels", [(40, 7, 0), (64, 20, 5), (33, 33, 3), (50, 49, 2)])
def test_select_equals_brute_force(L, b, levels):
    rng = np.random.default_rng(L + b)
    s = rng.integers(0, levels, L).astype(float) if levels else rng.standard_normal(L)
    want = brute.topk_indices(list(s), list(range(L)), b)
    np.testing.assert_array_equal(omnikv.select(s, b), want)


def _units(rng, Hkv, L, d):
    return [new_unit(rng.standard_normal((L, d)), rng.standard_normal((L, d)), np.arange(L)) for _ in range(Hkv)]


def test_paper_reuse_example():
    # The paper's example: an observation layer selects positions {1, 4, 8}
    # (1-based) and each sparse layer reads those positions from its own cache.
    # Eight positions after the step's append; J = {0, 3, 7} 0-based.  The sparse
    # layer's output must be dense attention over its own rows 0, 3, 7.
    rng = np.random.default_rng(3)
    Hkv, G, d, scale = 2, 2, 8, 0.35
    units = _units(rng, Hkv, 7, d)
    q = rng.standard_normal((Hkv * G, d))
    k_new, v_new = rng.standard_normal((Hkv, d)), rng.standard_normal((Hkv, d))
    J = np.array([0, 3, 7])
    res = omnikv.sparse_step(units, q, k_new, v_new, 7, scale, J)
    for a in range(Hkv * G):
        st = units[a // G]
        o, _, lse = brute.dense_attention(list(q[a]), [list(st.K[j]) for j in J], [list(st.V[j]) for j in J], scale)
        np.testing.assert_allclose(res["o"][a], o, rtol=0, atol=1e-12)
        assert abs(res["lse"][a] - lse) < 1e-12


def test_filter_step_is_dense_and_selection_uses_every_head():
    rng = np.random.default_rng(5)
    Hkv, G, d, scale, L = 2, 4, 16, 0.25, 30
    units = _units(rng, Hkv, L, d)
    q = rng.standard_normal((Hkv * G, d))
    k_new, v_new = rng.standard_normal((Hkv, d)), rng.standard_normal((Hkv, d))
    res = omnikv.filter_step(units, q, k_new, v_new, L, scale, 9)
    assert units[0].length == L + 1
    for a in range(Hkv * G):
        st = units[a // G]
        o, _, _ = brute.dense_attention(list(q[a]), [list(r) for r in st.K], [list(r) for r in st.V], scale)
        np.testing.assert_allclose(res["o"][a], o, rtol=0, atol=1e-12)
    # s by explicit loops over heads and positions (pure Python)
    for j in range(L + 1):
        want = max(scale * sum(float(x) * float(y) for x, y in zip(q[a], units[a // G].K[j])) for a in range(Hkv * G))
        assert abs(res["s"][j] - want) < 1e-12
    assert len(res["J"]) == 9 and np.all(np.diff(res["J"]) > 0)


def test_budget_covering_everything_is_dense():
    rng = np.random.default_rng(9)
    Hkv, G, d, scale, L = 1, 4, 8, 0.3, 12
    filt, sparse = _units(rng, Hkv, L, d), _units(rng, Hkv, L, d)
    q = rng.standard_normal((G, d))
    kn, vn = rng.standard_normal((Hkv, d)), rng.standard_normal((Hkv, d))
    J = omnikv.filter_step(filt, q, kn, vn, L, scale, 100)["J"]
    np.testing.assert_array_equal(J, np.arange(L + 1))
    res = omnikv.sparse_step(sparse, q, kn, vn, L, scale, J)
    st = sparse[0]
    for a in range(G):
        o, _, _ = brute.dense_attention(list(q[a]), [list(r) for r in st.K], [list(r) for r in st.V], scale)
        np.testing.assert_allclose(res["o"][a], o, rtol=0, atol=1e-12)


def test_selection_does_not_depend_on_the_sparse_layer():
    # J comes from the observation layer only; two sparse layers with different
    # caches read the same slots.
    rng = np.random.default_rng(11)
    Hkv, G, d, scale, L = 2, 2, 8, 0.3, 20
    filt = _units(rng, Hkv, L, d)
    q = rng.standard_normal((Hkv * G, d))
    kn, vn = rng.standard_normal((Hkv, d)), rng.standard_normal((Hkv, d))
    J = omnikv.filter_step(filt, q, kn, vn, L, scale, 6)["J"]
    a, b = _units(rng, Hkv, L, d), _units(rng, Hkv, L, d)
    ra = omnikv.sparse_step(a, q, kn, vn, L, scale, J)
    rb = omnikv.sparse_step(b, q, kn, vn, L, scale, J)
    assert not np.allclose(ra["o"], rb["o"])       # own caches, own outputs
    J2 = omnikv.filter_step(_units(np.random.default_rng(11), Hkv, L, d), q, kn, vn, L, scale, 6)["J"]
    np.testing.assert_array_equal(J, J2)
