"""Pins of the oracle's dispatch, expert FFN, combine and visual drop (CPU only).

Dispatch is checked against a per-expert scan; "combine inverts dispatch"
with identity experts; the SwiGLU FFN against torch's float64 library
routines (a one-expert layer is a dense SwiGLU MLP); the visual drop against
explicit slicing.
"""

import numpy as np
import pytest
import scipy.special
import torch

import oracle


def _scan_dispatch(idx, E):
    # for each expert in turn, collect (token, slot) assignments in token order
    T, k = idx.shape
    order = []
    counts = []
    for e in range(E):
        rows = [i * k + j for i in range(T) for j in range(k) if idx[i, j] == e]
        order += rows
        counts.append(len(rows))
    return np.array(counts), np.array(order, dtype=np.int64)


@pytest.mark.parametrize("seed", range(4))
def test_dispatch_against_scan_and_invariants(seed):
    rng = np.random.default_rng(seed)
    T, E, k = 37, 9, 3
    idx = np.stack([rng.permutation(E)[:k] for _ in range(T)])
    counts, offsets, src_of_row, row_of_slot = oracle.dispatch(idx, E)
    c2, o2 = _scan_dispatch(idx, E)
    np.testing.assert_array_equal(counts, c2)
    np.testing.assert_array_equal(src_of_row, o2)
    assert offsets[0] == 0 and offsets[-1] == T * k
    np.testing.assert_array_equal(np.diff(offsets), counts)
    assert sorted(src_of_row) == list(range(T * k))  # a bijection
    np.testing.assert_array_equal(row_of_slot[src_of_row], np.arange(T * k))
    for e in range(E):  # rows of one expert ascend by token
        toks = src_of_row[offsets[e]:offsets[e + 1]] // k
        assert np.all(np.diff(toks) > 0)
        assert (idx.reshape(-1)[src_of_row[offsets[e]:offsets[e + 1]]] == e).all()


def test_dispatch_prefix_experts_only_and_empty():
    rng = np.random.default_rng(5)
    idx = np.stack([rng.permutation(5)[:2] for _ in range(20)])
    counts, offsets, _, _ = oracle.dispatch(idx, 12)
    assert (counts[5:] == 0).all() and offsets[-1] == 40
    c, o, s, r = oracle.dispatch(np.zeros((0, 4), int), 7)
    assert c.sum() == 0 and o[-1] == 0 and len(s) == 0 and len(r) == 0


def test_combine_inverts_dispatch_with_identity_experts():
    rng = np.random.default_rng(6)
    T, E, k, d = 30, 8, 3, 5
    x = rng.standard_normal((T, d))
    idx = np.stack([rng.permutation(E)[:k] for _ in range(T)])
    _, _, src_of_row, row_of_slot = oracle.dispatch(idx, E)
    x_perm = x[src_of_row // k]  # identity expert: y_r = x_r
    # unit weights: k x exactly
    np.testing.assert_array_equal(oracle.combine(x_perm, row_of_slot, np.ones((T, k))), k * x)
    # weights summing to one: x back
    w = rng.dirichlet(np.ones(k), size=T)
    np.testing.assert_allclose(oracle.combine(x_perm, row_of_slot, w), x, rtol=1e-14, atol=1e-14)


def test_silu_matches_library():
    z = np.linspace(-30, 30, 1001)
    np.testing.assert_allclose(oracle.silu(z), z * scipy.special.expit(z), rtol=1e-14, atol=1e-300)
    zt = torch.from_numpy(z)
    np.testing.assert_allclose(oracle.silu(z), torch.nn.functional.silu(zt).numpy(), rtol=1e-14, atol=1e-300)


def test_one_expert_layer_is_dense_swiglu_mlp():
    """E = 1, k = 1: every token goes to the single expert with weight 1, so
    the layer is a dense SwiGLU MLP, computed here with torch float64 ops."""
    rng = np.random.default_rng(7)
    T, d, m = 19, 12, 7
    x = rng.standard_normal((T, d))
    wgu = rng.standard_normal((1, 2 * m, d)) * 0.4
    wd = rng.standard_normal((1, d, m)) * 0.4
    res = oracle.moe_layer_dense(x, rng.standard_normal((d, 1)), None, wgu, wd, 1)
    xt = torch.from_numpy(x)
    g = torch.nn.functional.linear(xt, torch.from_numpy(wgu[0, :m]))
    u = torch.nn.functional.linear(xt, torch.from_numpy(wgu[0, m:]))
    ref = torch.nn.functional.linear(torch.nn.functional.silu(g) * u, torch.from_numpy(wd[0]))
    np.testing.assert_allclose(res["out"], ref.numpy(), rtol=1e-12, atol=1e-13)


def test_layer_against_torch_per_token_loop():
    """A whole dense layer recomputed token by token with torch float64
    library ops (linear, silu, topk on the logits, softmax of the selected)."""
    rng = np.random.default_rng(8)
    T, d, E, m, k = 23, 10, 7, 6, 3
    x = rng.standard_normal((T, d))
    w_r = rng.standard_normal((d, E))
    b = rng.standard_normal(E)
    wgu = rng.standard_normal((E, 2 * m, d)) * 0.3
    wd = rng.standard_normal((E, d, m)) * 0.3
    res = oracle.moe_layer_dense(x, w_r, b, wgu, wd, k)
    F = torch.nn.functional
    for i in range(T):
        xi = torch.from_numpy(x[i])
        logit = xi @ torch.from_numpy(w_r) + torch.from_numpy(b)
        v, e_sel = torch.topk(logit, k)  # no exact ties in continuous data
        wt = torch.softmax(v, 0)
        acc = torch.zeros(d, dtype=torch.float64)
        for j in range(k):
            e = int(e_sel[j])
            gu = F.linear(xi, torch.from_numpy(wgu[e]))
            acc += wt[j] * F.linear(F.silu(gu[:m]) * gu[m:], torch.from_numpy(wd[e]))
        assert list(res["idx"][i]) == [int(t) for t in e_sel]
        np.testing.assert_allclose(res["out"][i], acc.numpy(), rtol=1e-11, atol=1e-12)


def test_drop_visual_block():
    h = np.arange(40.0).reshape(10, 4)
    np.testing.assert_array_equal(oracle.drop_visual_block(h, 0, 7), h[7:])
    np.testing.assert_array_equal(oracle.drop_visual_block(h, 3, 3), h)
    np.testing.assert_array_equal(oracle.drop_visual_block(h, 2, 10), h[:2])
    np.testing.assert_array_equal(oracle.drop_visual_block(h, 2, 5), h[[0, 1, 5, 6, 7, 8, 9]])
    with pytest.raises(ValueError):
        oracle.drop_visual_block(h, 5, 4)
