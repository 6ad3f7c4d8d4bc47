"""Pins for oracle.attention (CPU only)."""
import json
import math
import os

import numpy as np
import pytest

from oracle import attention, brute

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rand(rng, *shape):
    return rng.standard_normal(shape)


def test_two_slot_closed_form():
    g = json.load(open(os.path.join(GOLDEN, "attention_two_slot.json")))
    o, lse, alpha, z = attention.selected_attention(
        np.array(g["q"]), np.array(g["K"]), np.array(g["V"]), np.array(g["S"]), g["scale"])
    np.testing.assert_allclose(alpha, g["expect_alpha"], rtol=0, atol=1e-15)
    np.testing.assert_allclose(o, g["expect_o"], rtol=0, atol=1e-14)
    np.testing.assert_allclose(lse, g["expect_lse"], rtol=0, atol=1e-15)


@pytest.mark.parametrize("seed", range(6))
def test_dense_matches_pure_python(seed):
    rng = np.random.default_rng(seed)
    G, L, d = 4, int(rng.integers(1, 40)), 8
    q, K, V = _rand(rng, G, d), _rand(rng, L, d), _rand(rng, L, d)
    scale = 1.0 / math.sqrt(d)
    o, lse, alpha, _ = attention.selected_attention(q, K, V, np.arange(L), scale)
    for a in range(G):
        ob, wb, lb = brute.dense_attention(list(q[a]), K.tolist(), V.tolist(), scale)
        np.testing.assert_allclose(o[a], ob, rtol=0, atol=1e-12)
        np.testing.assert_allclose(alpha[a], wb, rtol=0, atol=1e-13)
        assert abs(lse[a] - lb) < 1e-12


def test_subset_equals_dense_over_subset():
    # Appendix A.1: sparse attention normalises over the selected positions
    # only; reading {1,4,8} of eight tokens equals dense attention over those three.
    rng = np.random.default_rng(7)
    d = 8
    q, K, V = _rand(rng, 1, d), _rand(rng, 8, d), _rand(rng, 8, d)
    S = np.array([0, 3, 7])
    o, _, alpha, _ = attention.selected_attention(q, K, V, S, 0.3)
    ob, wb, _ = brute.dense_attention(list(q[0]), K[S].tolist(), V[S].tolist(), 0.3)
    np.testing.assert_allclose(o[0], ob, atol=1e-13)
    np.testing.assert_allclose(alpha[0], wb, atol=1e-14)


def test_weights_sum_to_one_and_special_cases():
    rng = np.random.default_rng(3)
    d = 16
    q, K, V = _rand(rng, 4, d), _rand(rng, 30, d), _rand(rng, 30, d)
    _, _, alpha, _ = attention.selected_attention(q, K, V, np.arange(30), 0.25)
    np.testing.assert_allclose(alpha.sum(axis=1), 1.0, atol=1e-14)
    # A single slot returns its value.
    o1, lse1, a1, z1 = attention.selected_attention(q, K[:1], V[:1], np.array([0]), 0.25)
    np.testing.assert_array_equal(o1, np.repeat(V[:1], 4, axis=0))
    np.testing.assert_allclose(lse1, z1[:, 0], atol=0)
    # A zero query weights every slot equally: the mean of the values.
    o0, _, a0, _ = attention.selected_attention(np.zeros((1, d)), K, V, np.arange(30), 0.25)
    np.testing.assert_allclose(o0[0], V.mean(axis=0), atol=1e-14)


def test_permutation_invariance():
    rng = np.random.default_rng(11)
    q, K, V = _rand(rng, 2, 8), _rand(rng, 20, 8), _rand(rng, 20, 8)
    perm = rng.permutation(20)
    o, lse, _, _ = attention.selected_attention(q, K, V, np.arange(20), 0.5)
    o2, lse2, _, _ = attention.selected_attention(q, K[perm], V[perm], np.arange(20), 0.5)
    np.testing.assert_allclose(o, o2, atol=1e-14)
    np.testing.assert_allclose(lse, lse2, atol=1e-14)


def test_rejects_empty_or_repeated_read_set():
    K = np.zeros((3, 2))
    with pytest.raises(ValueError):
        attention.selected_attention(np.zeros((1, 2)), K, K, np.array([], dtype=np.int64), 1.0)
    with pytest.raises(ValueError):
        attention.selected_attention(np.zeros((1, 2)), K, K, np.array([1, 1]), 1.0)


def test_gqa_group_map():
    # g(a) = floor(a / G): KV head 2 with G = 4 serves query heads 8..11.
    np.testing.assert_array_equal(attention.group_heads(2, 4), [8, 9, 10, 11])
