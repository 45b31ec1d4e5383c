"""Property-based pins of the oracle (hypothesis, bounded examples): the
invariants the paper's definitions fix, checked over random small shapes
against brute force written independently of the oracle's code paths.

- Top-k routing (Eq. 10): the selected experts are k distinct indices whose
  logits are not exceeded by any unselected one (ties to the lower index),
  and the renormalised weights sum to 1.
- Prefix length (Eq. 12): K is the first K whose running mass reaches
  p * total, found here by trying every K; K >= k.
- Prefix re-route (Sec. 3.3): every selected expert lies below K and the
  weights equal the softmax over the selected logits.
- Dispatch and combine: the grouping is the stable sort of the assignments
  by expert, and combine with unit experts (y row = token row) returns the
  weighted sum of each token's own row.
"""

import itertools

import numpy as np
import pytest
from hypothesis import given, settings
from hypothesis import strategies as st

import oracle

pytestmark = pytest.mark.filterwarnings("ignore")

SETTINGS = settings(max_examples=60, deadline=None, derandomize=True)


@st.composite
def logits_case(draw):
    T = draw(st.integers(1, 6))
    E = draw(st.integers(1, 9))
    k = draw(st.integers(1, E))
    # few distinct values so that ties occur
    vals = draw(st.lists(st.sampled_from([-2.0, -0.5, 0.0, 0.25, 1.0, 3.0]), min_size=T * E, max_size=T * E))
    return np.array(vals, np.float64).reshape(T, E), k


@SETTINGS
@given(logits_case())
def test_topk_selection_and_weights(case):
    a, k = case
    T, E = a.shape
    idx, w = oracle.full_pool_route(a, k)
    for i in range(T):
        sel = [int(e) for e in idx[i]]
        assert len(set(sel)) == k and all(0 <= e < E for e in sel)
        # brute force: the k best (value descending, index ascending)
        best = sorted(range(E), key=lambda e: (-a[i, e], e))[:k]
        assert sel == best
        assert abs(w[i].sum() - 1.0) < 1e-12
        ex = np.exp(a[i, sel] - a[i, sel].max())
        np.testing.assert_allclose(w[i], ex / ex.sum(), rtol=1e-12, atol=0)


@st.composite
def mass_case(draw):
    E = draw(st.integers(1, 10))
    k = draw(st.integers(1, E))
    s = np.array(draw(st.lists(st.sampled_from([0.0, 0.125, 0.5, 1.0, 2.0, 3.5]), min_size=E, max_size=E)),
                 np.float64)
    p = draw(st.sampled_from([0.05, 0.25, 0.5, 0.75, 0.9, 1.0]))
    return s, p, k


@SETTINGS
@given(mass_case())
def test_prefix_length_is_first_covering_prefix(case):
    s, p, k = case
    E = s.size
    K = oracle.prefix_length(s, p, k)
    tot = sum(float(v) for v in s)
    run, k_hat = 0.0, E
    for j in range(E):  # try every K in order
        run += float(s[j])
        if run >= p * tot:
            k_hat = j + 1
            break
    assert K == max(k, k_hat)
    assert k <= K <= E


@SETTINGS
@given(logits_case(), st.integers(0, 8))
def test_prefix_reroute_stays_inside_prefix(case, extra):
    a, k = case
    T, E = a.shape
    K = min(E, k + extra)
    idx, w = oracle.prefix_route(a, K, k)
    for i in range(T):
        sel = [int(e) for e in idx[i]]
        assert all(0 <= e < K for e in sel) and len(set(sel)) == k
        best = sorted(range(K), key=lambda e: (-a[i, e], e))[:k]
        assert sel == best
        ex = np.exp(a[i, sel] - a[i, sel].max())
        np.testing.assert_allclose(w[i], ex / ex.sum(), rtol=1e-12, atol=0)


@st.composite
def routing_case(draw):
    T = draw(st.integers(0, 7))
    E = draw(st.integers(1, 6))
    k = draw(st.integers(1, E))
    rows = [draw(st.permutations(range(E)))[:k] for _ in range(T)]
    idx = np.array(rows, np.int64).reshape(T, k)
    w = np.array(draw(st.lists(st.floats(0.0, 1.0), min_size=T * k, max_size=T * k)), np.float64).reshape(T, k)
    return idx, w, E


@SETTINGS
@given(routing_case())
def test_dispatch_is_stable_sort_and_combine_inverts_it(case):
    idx, w, E = case
    T, k = idx.shape
    counts, offsets, src, ros = oracle.dispatch(idx, E)
    A = T * k
    flat = idx.reshape(-1)
    expect = sorted(range(A), key=lambda a: (flat[a], a))  # stable by expert
    assert list(src) == expect
    assert sorted(src) == list(range(A))
    assert all(ros[src[r]] == r for r in range(A))
    assert list(counts) == [int((flat == e).sum()) for e in range(E)]
    assert list(offsets) == [0] + list(itertools.accumulate(counts))
    # unit experts: dispatched row r carries its token's row
    x = np.arange(T * 3, dtype=np.float64).reshape(T, 3) + 1.0
    y = x[np.asarray(src) // k] if A else np.zeros((0, 3))
    out = oracle.combine(y, ros, w)
    np.testing.assert_allclose(out, w.sum(axis=1, keepdims=True) * x if T else out, rtol=1e-12, atol=0)
