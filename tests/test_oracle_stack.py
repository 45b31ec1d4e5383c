"""Pins of the oracle's stack of MoE blocks (Algorithm 2's loop over layers
with the residual stream), CPU only.

  * zero down projections make every block the identity, so the stack
    returns the input with the visual rows removed, and K is reported only
    for the layers from the exit on;
  * dense blocks route per token, so before the exit the text rows do not
    depend on the visual rows: the stack over visual + text rows equals the
    stack over the text rows alone (a drop placed one layer late, or RCEP
    run over the visual rows, changes K and fails this);
  * at p = 1 with every expert routed, K = E and the RCEP block is the dense
    block (Eq. 12), so the text rows equal those of the all-dense stack.
  * the component-ablation modes (Table 2): the exit alone ("dense" after the
    exit) keeps the text rows of the stack without an exit, since a dense
    block routes each token by itself; a fixed prefix of E is the full pool;
    a fixed prefix equal, layer by layer, to the K that Eq. 12 chose
    reproduces the RCEP stack; and a fixed prefix below k is rejected.
"""

import numpy as np
import pytest

import oracle

D, E, M, K_TOP = 16, 6, 8, 2


def _layers(n, seed, zero_down=False):
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(n):
        out.append(dict(
            w_r=rng.normal(0, 0.5, (D, E)),
            bias=rng.normal(0, 0.5, E),
            w_gate_up=rng.normal(0, 0.3, (E, 2 * M, D)),
            w_down=np.zeros((E, D, M)) if zero_down else rng.normal(0, 0.3, (E, D, M)),
        ))
    return out


def test_zero_blocks_leave_the_kept_rows():
    rng = np.random.default_rng(0)
    h = rng.normal(size=(12, D))
    out, Ks = oracle.moe_stack(h, _layers(4, 1, zero_down=True), K_TOP, 0.8, exit_layer=2, v0=0,
                               v1=8)
    np.testing.assert_array_equal(out, h[8:])
    assert Ks[0] is None and Ks[1] is None
    assert all(K is not None and K_TOP <= K[0] <= E for K in Ks[2:])
    # a visual block in the middle of the rows
    out, _ = oracle.moe_stack(h, _layers(3, 1, zero_down=True), K_TOP, 0.8, exit_layer=1, v0=3,
                              v1=7)
    np.testing.assert_array_equal(out, np.concatenate([h[:3], h[7:]]))


@pytest.mark.parametrize("seed", [3, 7])
def test_text_rows_do_not_see_the_visual_rows(seed):
    rng = np.random.default_rng(seed)
    vis, txt = rng.normal(size=(24, D)) * 3.0, rng.normal(size=(8, D))
    layers = _layers(4, seed + 10)
    out, Ks = oracle.moe_stack(np.concatenate([vis, txt]), layers, K_TOP, 0.7, exit_layer=2, v0=0,
                               v1=24)
    ref, Ks_ref = oracle.moe_stack(txt, layers, K_TOP, 0.7, exit_layer=2)
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-12)
    assert [int(K[0]) for K in Ks[2:]] == [int(K[0]) for K in Ks_ref[2:]]
    # the pin has power: prefix lengths computed over visual + text rows
    # (an exit one layer late) differ for these inputs
    h = np.concatenate([vis, txt])
    for prm in layers[:2]:
        h = h + oracle.moe_layer_dense(h, prm["w_r"], prm["bias"], prm["w_gate_up"],
                                       prm["w_down"], K_TOP)["out"]
    late = oracle.moe_layer_rcep(h, layers[2]["w_r"], layers[2]["bias"], layers[2]["w_gate_up"],
                                 layers[2]["w_down"], K_TOP, 0.7)["K"]
    assert int(late[0]) != int(Ks[2][0])


def test_p_one_with_full_support_is_the_dense_stack():
    rng = np.random.default_rng(4)
    h = rng.normal(size=(40, D))
    layers = _layers(3, 5)
    out, Ks = oracle.moe_stack(h, layers, K_TOP, 1.0, exit_layer=1, v0=0, v1=8)
    assert all(int(K[0]) == E for K in Ks[1:])  # every expert routed
    dense, Kd = oracle.moe_stack(h, layers, K_TOP, 1.0, exit_layer=None)
    assert all(K is None for K in Kd)
    np.testing.assert_allclose(out, dense[8:], rtol=0, atol=1e-12)


def test_exit_alone_keeps_the_text_rows_of_the_dense_stack():
    rng = np.random.default_rng(8)
    h = rng.normal(size=(30, D))
    layers = _layers(4, 9)
    out, Ks = oracle.moe_stack(h, layers, K_TOP, 0.7, exit_layer=2, v0=0, v1=10, after_exit="dense")
    assert all(K is None for K in Ks)
    dense, _ = oracle.moe_stack(h, layers, K_TOP, 0.7, exit_layer=None)
    np.testing.assert_allclose(out, dense[10:], rtol=0, atol=1e-12)
    # the mode has power: RCEP after the exit prunes experts and moves the rows
    rc, Kr = oracle.moe_stack(h, layers, K_TOP, 0.7, exit_layer=2, v0=0, v1=10)
    assert any(int(K[0]) < E for K in Kr[2:])
    assert np.abs(rc - out).max() > 1e-6


def test_fixed_prefix_modes():
    rng = np.random.default_rng(12)
    h = rng.normal(size=(26, D))
    layers = _layers(4, 13)
    full, Kf = oracle.moe_stack(h, layers, K_TOP, 0.6, exit_layer=1, v0=0, v1=6, after_exit="fixed",
                                K_fixed=E)
    assert all(int(K[0]) == E for K in Kf[1:])
    ex, _ = oracle.moe_stack(h, layers, K_TOP, 0.6, exit_layer=1, v0=0, v1=6, after_exit="dense")
    np.testing.assert_allclose(full, ex, rtol=0, atol=1e-12)
    rc, Kr = oracle.moe_stack(h, layers, K_TOP, 0.6, exit_layer=1, v0=0, v1=6)
    per_layer = [0] + [int(K[0]) for K in Kr[1:]]
    assert min(per_layer[1:]) < E  # Eq. 12 prunes somewhere
    fx, Kx = oracle.moe_stack(h, layers, K_TOP, 0.6, exit_layer=1, v0=0, v1=6, after_exit="fixed",
                              K_fixed=per_layer)
    np.testing.assert_array_equal(fx, rc)
    assert [int(K[0]) for K in Kx[1:]] == per_layer[1:]
    # a shorter fixed prefix routes inside it only
    short, Ks = oracle.moe_stack(h, layers, K_TOP, 0.6, exit_layer=1, v0=0, v1=6, after_exit="fixed",
                                 K_fixed=3)
    assert all(int(K[0]) == 3 for K in Ks[1:])
    assert np.abs(short - rc).max() > 1e-6
    with pytest.raises(ValueError):
        oracle.moe_stack(h, layers, K_TOP, 0.6, exit_layer=1, v0=0, v1=6, after_exit="fixed", K_fixed=1)
    with pytest.raises(ValueError):
        oracle.moe_stack(h, layers, K_TOP, 0.6, exit_layer=1, after_exit="fixed")
