"""Pins of the oracle's router, Top-k and renormalised weights (CPU only).

Each check is independent of the oracle's own code path: exhaustive subset
search, selection by scanning, closed forms, library softmax, and the
paper's structural statements (Sec. 3.3, Algorithm 2).
"""

import itertools
import json
import math
import os

import numpy as np
import pytest
import scipy.special

import oracle

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _select_scan(row, k):
    """Top-k by repeated scanning: the largest remaining value, lowest index on ties."""
    left = list(range(len(row)))
    out = []
    for _ in range(k):
        best = left[0]
        for e in left[1:]:
            if row[e] > row[best]:
                best = e
        out.append(best)
        left.remove(best)
    return out


@pytest.mark.parametrize("seed", range(6))
def test_topk_matches_scan_and_exhaustive_subsets(seed):
    rng = np.random.default_rng(seed)
    for _ in range(40):
        T, E = rng.integers(1, 9), rng.integers(1, 7)
        k = int(rng.integers(1, E + 1))
        a = rng.integers(-2, 3, size=(T, E)).astype(np.float64)  # many exact ties
        idx = oracle.topk_by_logit(a, k)
        for i in range(T):
            assert list(idx[i]) == _select_scan(a[i], k)
            # the chosen set maximises the sum of logits over every k-subset
            best = max(sum(a[i, list(c)]) for c in itertools.combinations(range(E), k))
            assert sum(a[i, idx[i]]) == best


def test_topk_on_logits_equals_topk_on_probabilities():
    # softmax is strictly increasing, so TopK(q) of Eq. 10 equals TopK(a)
    rng = np.random.default_rng(7)
    a = rng.standard_normal((300, 128))
    q = oracle.softmax(a)
    np.testing.assert_array_equal(oracle.topk_by_logit(a, 8), oracle.topk_by_logit(q, 8))


def test_softmax_matches_library():
    rng = np.random.default_rng(1)
    a = rng.standard_normal((17, 33)) * 4
    np.testing.assert_allclose(oracle.softmax(a), scipy.special.softmax(a, axis=1), rtol=1e-13, atol=0)


def test_weights_sum_to_one_and_equal_softmax_of_selected_logits():
    rng = np.random.default_rng(2)
    a = rng.standard_normal((64, 32)) * 3
    idx, w = oracle.full_pool_route(a, 5)
    np.testing.assert_allclose(w.sum(1), 1.0, rtol=0, atol=1e-14)
    sel = np.take_along_axis(a, idx, 1)
    np.testing.assert_allclose(w, scipy.special.softmax(sel, axis=1), rtol=1e-12, atol=0)
    # slots are stored by descending logit, so weights are non-increasing
    assert np.all(np.diff(w, axis=1) <= 1e-15)


def test_all_equal_logits():
    a = np.full((3, 10), 0.25)
    idx, w = oracle.full_pool_route(a, 4)
    assert (idx == np.arange(4)).all()
    np.testing.assert_allclose(w, 0.25, rtol=0, atol=1e-15)


def test_decreasing_logits_golden():
    g = json.load(open(os.path.join(GOLD, "decreasing_logits_weights.json")))
    a = np.array([g["logits"]])
    idx, w = oracle.full_pool_route(a, g["k"])
    assert list(idx[0]) == g["idx"]
    np.testing.assert_allclose(w[0], g["w"], rtol=1e-15, atol=0)


def test_router_logits_special_cases():
    rng = np.random.default_rng(3)
    E = 6
    x = rng.standard_normal((5, E))
    b = rng.standard_normal(E)
    # identity router weights: logits = x + b  (a dropped bias or a transposed
    # weight would fail one of these)
    np.testing.assert_allclose(oracle.router_logits(x, np.eye(E), b), x + b, rtol=0, atol=1e-15)
    w = rng.standard_normal((E, 3 * E))[:, :E]
    np.testing.assert_allclose(oracle.router_logits(np.zeros((2, E)), w, b), np.tile(b, (2, 1)), atol=0)
    # a single one-hot token row picks one row of W_r
    xo = np.zeros((1, E))
    xo[0, 2] = 1.0
    w2 = rng.standard_normal((E, 4))
    np.testing.assert_allclose(oracle.router_logits(xo, w2)[0], w2[2], atol=0)


def test_prefix_route_K_equal_E_is_full_pool():
    rng = np.random.default_rng(4)
    a = rng.standard_normal((50, 16))
    i1, w1 = oracle.full_pool_route(a, 4)
    i2, w2 = oracle.prefix_route(a, 16, 4)
    np.testing.assert_array_equal(i1, i2)
    np.testing.assert_allclose(w1, w2, rtol=1e-14)


def test_prefix_route_keeps_tokens_already_inside_prefix():
    rng = np.random.default_rng(5)
    a = rng.standard_normal((400, 16))
    K, k = 9, 3
    i_full, w_full = oracle.full_pool_route(a, k)
    i_pre, w_pre = oracle.prefix_route(a, K, k)
    inside = (i_full < K).all(1)
    assert inside.any() and (~inside).any()
    np.testing.assert_array_equal(i_full[inside], i_pre[inside])
    np.testing.assert_allclose(w_full[inside], w_pre[inside], rtol=1e-13)
    # everything lies inside the prefix, k distinct experts per token
    assert (i_pre < K).all()
    assert all(len(set(r)) == k for r in i_pre)


def test_prefix_route_is_not_an_intersection():
    # full-pool top-2 of the token is {3, 0}; with K = 2 the new Top-2 inside
    # the prefix is {0, 1}: two experts, not the intersection {0}
    a = np.array([[1.0, 0.5, -1.0, 2.0]])
    idx, w = oracle.prefix_route(a, 2, 2)
    assert list(idx[0]) == [0, 1]
    e = np.exp([1.0, 0.5])
    np.testing.assert_allclose(w[0], e / e.sum(), rtol=1e-15)


def test_prefix_route_uses_new_softmax_over_prefix():
    rng = np.random.default_rng(6)
    a = rng.standard_normal((20, 12))
    K, k = 7, 3
    idx, w = oracle.prefix_route(a, K, k)
    qt = scipy.special.softmax(a[:, :K], axis=1)
    for i in range(20):
        sel = qt[i, idx[i]]
        np.testing.assert_allclose(w[i], sel / sel.sum(), rtol=1e-13)
        assert list(idx[i]) == _select_scan(a[i, :K], k)


def test_prefix_route_rejects_K_below_k():
    with pytest.raises(ValueError):
        oracle.prefix_route(np.zeros((1, 8)), 2, 3)


def test_reorder_does_not_change_dense_layer():
    """Sec. 3.3 and Algorithm 1: applying pi to the router outputs and the
    expert tensors changes storage, not the function of the unsliced layer."""
    rng = np.random.default_rng(8)
    T, d, E, m, k = 24, 8, 6, 5, 2
    x = rng.standard_normal((T, d))
    w_r = rng.standard_normal((d, E))
    b = rng.standard_normal(E)
    wgu = rng.standard_normal((E, 2 * m, d)) * 0.3
    wd = rng.standard_normal((E, d, m)) * 0.3
    ref = oracle.moe_layer_dense(x, w_r, b, wgu, wd, k)["out"]
    pi = rng.permutation(E)
    out = oracle.moe_layer_dense(x, *oracle.permute_experts(pi, w_r, b, wgu, wd), k)["out"]
    np.testing.assert_allclose(out, ref, rtol=1e-12, atol=1e-12)
