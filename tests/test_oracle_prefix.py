"""Pins of the oracle's masses, calibration order and prefix length (CPU only).

Eqs. 8, 9, 11 and 12 of the paper.  Checks: a hand-worked example at exact
equality, brute force over every prefix and over every expert subset,
invariants (total mass, monotonicity in p, K >= k, K(1) = last positive
expert) and a dense-matrix recomputation of the masses.
"""

import itertools
import json
import os

import numpy as np
import pytest

import oracle

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _dense_mass(idx, w, E):
    # the T x E matrix of renormalised weights (zero off the Top-k set), column sums
    T = idx.shape[0]
    dense = np.zeros((T, E))
    for i in range(T):
        for j in range(idx.shape[1]):
            dense[i, idx[i, j]] = w[i, j]
    return dense.sum(0)


def test_worked_example_golden():
    g = json.load(open(os.path.join(GOLD, "prefix_worked_example.json")))
    idx, w = np.array(g["topk_idx"]), np.array(g["topk_w"])
    s = oracle.activated_mass(idx, w, g["E"])
    np.testing.assert_array_equal(s, g["mass"])
    for c in g["cases"]:
        assert oracle.prefix_length(s, c["p"], g["k"]) == c["K"], c["why"]
    rr = g["prefix_reroute_at_p_0.75"]
    i2, w2 = oracle.prefix_route(np.array(rr["logits"]), 1, 1)
    np.testing.assert_array_equal(i2, rr["idx"])
    np.testing.assert_array_equal(w2, rr["w"])


@pytest.mark.parametrize("seed", range(4))
def test_mass_invariants_and_dense_recount(seed):
    rng = np.random.default_rng(seed)
    T, E, k = 200, 16, 3
    a = rng.standard_normal((T, E)) * 2
    idx, w = oracle.full_pool_route(a, k)
    s = oracle.activated_mass(idx, w, E)
    np.testing.assert_allclose(s, _dense_mass(idx, w, E), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(s.sum(), T, rtol=1e-12)  # each token contributes 1
    M = oracle.routed_mass(idx, w, E)
    np.testing.assert_allclose(M.sum(), 1.0, rtol=1e-12)


def _brute_K(s, p, k):
    E = len(s)
    tot = sum(s)
    ok = [K for K in range(1, E + 1) if sum(s[:K]) >= p * tot]
    return max(k, min(ok))


@pytest.mark.parametrize("seed", range(5))
def test_prefix_length_brute_force_and_bracket(seed):
    rng = np.random.default_rng(seed)
    for _ in range(200):
        E = int(rng.integers(1, 12))
        k = int(rng.integers(1, E + 1))
        s = rng.integers(0, 5, size=E).astype(float) * rng.choice([0.25, 0.5, 1.0])
        p = float(rng.choice([0.1, 0.25, 0.5, 0.7, 0.75, 0.9, 1.0, rng.uniform(0.01, 1)]))
        K = oracle.prefix_length(s, p, k)
        assert K == _brute_K(list(s), p, k)
        assert k <= K <= E
        c = np.cumsum(s)
        if s.sum() > 0:
            kh = int(np.argmax(c >= p * c[-1])) + 1  # first prefix reaching p
            assert c[kh - 1] >= p * c[-1]
            if kh > 1:
                assert c[kh - 2] < p * c[-1]


def test_prefix_length_monotone_in_p_and_limits():
    rng = np.random.default_rng(11)
    for _ in range(50):
        E, k = 32, 4
        s = np.sort(rng.exponential(size=E))[::-1]
        s[rng.integers(E // 2, E):] = 0.0  # a zero-mass tail
        ps = np.linspace(0.01, 1.0, 60)
        Ks = [oracle.prefix_length(s, p, k) for p in ps]
        assert all(a <= b for a, b in zip(Ks, Ks[1:]))
        # K(1.0) is the position of the last positive-mass expert (or k)
        last = int(np.nonzero(s > 0)[0].max()) + 1
        assert oracle.prefix_length(s, 1.0, k) == max(k, last)
        # small p gives K = k (the clamp of Eq. 12)
        assert oracle.prefix_length(s, 1e-6, k) == k


def test_prefix_length_empty_invocation_and_bad_p():
    assert oracle.prefix_length(np.zeros(8), 0.9, 3) == 3
    for bad in (0.0, -0.1, 1.0000001):
        with pytest.raises(ValueError):
            oracle.prefix_length(np.ones(4), bad, 1)


def test_prefix_is_minimum_cardinality_cover_when_sorted():
    """When calibration and runtime use the same tokens the reordered mass is
    non-increasing, and the shortest covering prefix is then the smallest
    expert subset of any shape that covers p of the mass (16 experts: all
    2^16 subsets are enumerated)."""
    rng = np.random.default_rng(12)
    T, E, k = 256, 16, 2
    a = rng.standard_normal((T, E)) + rng.standard_normal(E) * 1.5
    idx, w = oracle.full_pool_route(a, k)
    pi, _ = oracle.mean_mass_order(oracle.routed_mass(idx, w, E)[None])
    a2 = a[:, pi]
    i2, w2 = oracle.full_pool_route(a2, k)
    s = oracle.activated_mass(i2, w2, E)
    assert np.all(np.diff(s) <= 1e-12)
    tot = s.sum()
    for p in (0.3, 0.6, 0.9, 0.97):
        K = oracle.prefix_length(s, p, 1)
        best = None
        for r in range(1, E + 1):
            if any(sum(s[list(c)]) >= p * tot - 1e-12 for c in itertools.combinations(range(E), r)):
                best = r
                break
        assert K == best


def test_mean_mass_order_descending_and_stable():
    M = np.array([[0.1, 0.3, 0.3, 0.0, 0.3, 0.0],
                  [0.3, 0.1, 0.1, 0.0, 0.5, 0.0]])
    pi, mean = oracle.mean_mass_order(M)
    np.testing.assert_allclose(mean, [0.2, 0.2, 0.2, 0.0, 0.4, 0.0])
    # ties keep the lower native index first
    assert list(pi) == [4, 0, 1, 2, 3, 5]
    assert sorted(pi) == list(range(6))


def test_mean_is_over_cases_not_tokens():
    # App. A.4: masses are averaged within a case first, then across cases,
    # so a long case does not dominate
    E, k = 3, 1
    idx_long = np.zeros((100, 1), int)  # 100 tokens all on expert 0
    idx_short = np.full((1, 1), 2)  # 1 token on expert 2
    w1 = np.ones((100, 1))
    w2 = np.ones((1, 1))
    M = np.stack([oracle.routed_mass(idx_long, w1, E), oracle.routed_mass(idx_short, w2, E)])
    pi, mean = oracle.mean_mass_order(M)
    np.testing.assert_allclose(mean, [0.5, 0.0, 0.5])
    assert list(pi) == [0, 2, 1]


def test_rcep_layer_with_p_one_and_full_support_equals_dense():
    rng = np.random.default_rng(13)
    T, d, E, m, k = 64, 8, 6, 4, 2
    x = rng.standard_normal((T, d))
    w_r = rng.standard_normal((d, E))
    wgu = rng.standard_normal((E, 2 * m, d)) * 0.3
    wd = rng.standard_normal((E, d, m)) * 0.3
    dense = oracle.moe_layer_dense(x, w_r, None, wgu, wd, k)
    rcep = oracle.moe_layer_rcep(x, w_r, None, wgu, wd, k, 1.0)
    assert (rcep["mass"][0] > 0).all() and rcep["K"][0] == E
    np.testing.assert_array_equal(rcep["idx"], dense["idx"])
    np.testing.assert_allclose(rcep["out"], dense["out"], rtol=1e-13, atol=1e-13)


def test_rcep_layer_segments_are_independent_invocations():
    rng = np.random.default_rng(14)
    T, d, E, m, k = 40, 8, 10, 4, 2
    x = rng.standard_normal((T, d))
    w_r = rng.standard_normal((d, E))
    wgu = rng.standard_normal((E, 2 * m, d)) * 0.3
    wd = rng.standard_normal((E, d, m)) * 0.3
    so = [0, 15, 15, 40]  # includes an empty segment
    res = oracle.moe_layer_rcep(x, w_r, None, wgu, wd, k, 0.6, seg_offsets=so)
    assert res["K"][1] == k
    for s in (0, 2):
        lo, hi = so[s], so[s + 1]
        one = oracle.moe_layer_rcep(x[lo:hi], w_r, None, wgu, wd, k, 0.6)
        assert one["K"][0] == res["K"][s]
        np.testing.assert_array_equal(one["idx"], res["idx"][lo:hi])
        np.testing.assert_allclose(one["out"], res["out"][lo:hi], rtol=1e-13, atol=1e-13)
