"""Stack parity: the 48-layer prefill (7680 visual + 512 text rows, exit at
layer 20, p = 0.9) and the 64-token decode through the same 48 layers
(p = 0.85, RCEP in every layer, replayed from a HIP graph), plus a tiny fp32
stack, against the oracle, and the two load-time and residual entry points
(moe_permute_experts, moe_combine_residual).

Protocol: teacher-forced per layer.  The GPU's input rows of layer l and
its float32 logits are widened to float64 and fed to the oracle's layer, so
expert indices and K compare bit for bit (K up to a declared near-tie).
The layer's MoE output (its combine without the residual) compares within
2e-2 (bf16) or 1e-4 (fp32) of the oracle's, relative to the max.  The
residual update h_{l+1} = h_l + out_l then compares within the same bound
plus half a unit in the last place of h_{l+1} (it is rounded once to the
storage precision).  Expert orders are checked against the oracle's
Mean-Mass order of the GPU's calibration routing.
"""

import numpy as np
import pytest
import torch

import oracle
from _util import ensure_built, rel_inf, row_rel

pytestmark = pytest.mark.gpu

from paper_2609_38823_amd import abi  # noqa: E402
from paper_2609_38823_amd import inputs as I  # noqa: E402
from paper_2609_38823_amd.layer import to_device  # noqa: E402
from paper_2609_38823_amd.stack import MoEStack  # noqa: E402

TOL = {"f32": 1e-4, "bf16": 2e-2}
EPS = {"f32": 2.0 ** -24, "bf16": 2.0 ** -9}  # unit roundoff (half an ulp, relative)


@pytest.fixture(scope="module", autouse=True)
def _lib():
    ensure_built()
    torch.cuda.init()


def host(t):
    torch.cuda.synchronize()
    return (t.float() if t.dtype == torch.bfloat16 else t).cpu().numpy()


def near_tie(mass, p, K, rel=1e-9):
    c = np.cumsum(np.asarray(mass, np.float64))
    tot, thr = c[-1], p * c[-1]
    m = min(abs(c[K - 1] - thr), abs(thr - c[K - 2]) if K >= 2 else np.inf)
    return m < rel * tot


# ---------------------------------------------------------------- entry points
@pytest.mark.parametrize("dt,E,d,m", [("bf16", 8, 64, 32), ("f32", 5, 24, 12), ("bf16", 3, 10, 7)])
def test_permute_experts_bitwise(dt, E, d, m):
    """moe_permute_experts moves storage only: bitwise numpy fancy indexing;
    an order entry outside [0, E) yields a zero expert."""
    rng = np.random.default_rng(E * 100 + d)
    tdt = torch.bfloat16 if dt == "bf16" else torch.float32
    w_r = rng.normal(size=(d, E)).astype(np.float32)
    bias = rng.normal(size=E).astype(np.float32)
    gu = torch.from_numpy(rng.normal(size=(E, 2 * m, d)).astype(np.float32)).cuda().to(tdt)
    dn = torch.from_numpy(rng.normal(size=(E, d, m)).astype(np.float32)).cuda().to(tdt)
    order = rng.permutation(E).astype(np.int32)
    bad = order.copy()
    bad[E // 2] = E + 3  # out of range -> zeros
    for o in (order, bad):
        out = [torch.full_like(t, 7) for t in (to_device(w_r, torch.float32),
                                               to_device(bias, torch.float32), gu, dn)]
        abi.moe_permute_experts(torch.from_numpy(o).cuda(), to_device(w_r, torch.float32),
                                to_device(bias, torch.float32), gu, dn, *out)
        ok = (o >= 0) & (o < E)
        src = np.where(ok, o, 0)
        exp = [w_r[:, src] * ok, bias[src] * ok, host(gu)[src] * ok[:, None, None],
               host(dn)[src] * ok[:, None, None]]
        for g, e in zip(out, exp):
            np.testing.assert_array_equal(host(g), e)


@pytest.mark.parametrize("dt,T,k,d", [("bf16", 300, 8, 2048), ("bf16", 77, 3, 136),
                                      ("f32", 129, 2, 256), ("bf16", 5, 2, 9), ("bf16", 20000, 2, 2048)])
@pytest.mark.parametrize("in_place", [False, True])
def test_combine_residual(dt, T, k, d, in_place):
    """out = residual + sum_j w_j y_row(j): against the oracle's combine plus
    the residual, out of place and in place (out is residual)."""
    rng = np.random.default_rng(T + d)
    tdt = torch.bfloat16 if dt == "bf16" else torch.float32
    rnd = I.round_to_bf16 if dt == "bf16" else (lambda a: a.astype(np.float32))
    A = T * k
    y = rnd(rng.normal(size=(A, d)).astype(np.float32))
    res = rnd(rng.normal(size=(T, d)).astype(np.float32))
    row_of_slot = rng.permutation(A).astype(np.int32)
    w = rng.uniform(0, 1, size=(T, k)).astype(np.float32)
    yd, rd = torch.from_numpy(y).cuda().to(tdt), torch.from_numpy(res).cuda().to(tdt)
    out = rd if in_place else torch.empty_like(rd)
    abi.moe_combine_residual(yd, torch.from_numpy(row_of_slot).cuda(), torch.from_numpy(w).cuda(),
                             rd, out)
    ref = res.astype(np.float64) + oracle.combine(y, row_of_slot, w)
    got = host(out)
    bound = TOL[dt] * np.abs(ref).max()
    assert np.abs(got - ref).max() <= bound
    if not in_place:
        np.testing.assert_array_equal(host(rd), res)  # residual untouched


# ---------------------------------------------------------------- stacks
def oracle_params(stack, l):
    """Layer l's parameters for the oracle: the generator's native weights
    (host copies), then the GPU's Mean-Mass order, applied by the oracle."""
    sh, wl = stack.sh, stack.wl
    rp = I.router_params(sh, wl.seed, l)
    gu, dn = I.device_expert_weights(sh, wl.seed, l)
    gu_h, dn_h = host(gu), host(dn)
    del gu, dn
    w_r, bias, wgu, wd = oracle.permute_experts(stack.orders[l], rp["w_r"], rp["bias"], gu_h, dn_h)
    return dict(w_r=w_r, bias=bias, w_gate_up=wgu, w_down=wd)


def check_order(stack, l):
    """The layer's order equals the oracle's Mean-Mass order (Eqs. 8, 9) of
    the GPU's full-pool routing of the calibration rows entering layer l
    (teacher-forced: the GPU's carried calibration rows)."""
    sh, wl = stack.sh, stack.wl
    rp = I.router_params(sh, wl.seed, l)
    xc = stack.calib_h[l]
    T, E = xc.shape[0], sh.E
    logits = torch.empty((T, E), dtype=torch.float32, device="cuda")
    idx = torch.empty((T, sh.k), dtype=torch.int32, device="cuda")
    w = torch.empty((T, sh.k), dtype=torch.float32, device="cuda")
    ws = torch.empty(abi.moe_workspace_size(T, E, sh.k, sh.d, 1, 1), dtype=torch.uint8, device="cuda")
    abi.moe_route(xc, to_device(rp["w_r"], torch.float32), to_device(rp["bias"], torch.float32), sh.k,
                  logits, idx, w, ws=ws)
    M = oracle.routed_mass(host(idx), host(w).astype(np.float64), E)
    np.testing.assert_array_equal(stack.orders[l], oracle.mean_mass_order(M[None, :])[0])


def check_layer(stack, l, h_in, rcep, p, dt, sample=None, K_fixed=None):
    """Run layer l on h_in through the stack's call, then compare it with the
    oracle's layer fed the same rows and the GPU's logits (K_fixed: a given
    prefix length instead of Eq. 12)."""
    h0 = host(h_in).copy()
    dst = torch.empty_like(h_in)
    b = stack.layer_forward(l, h_in, dst, rcep, p, K_fixed=K_fixed)
    # the layer's MoE output on its own (same y_perm, rows and weights)
    abi.moe_combine(b.y_perm, b.row_of_slot, b.w, b.out)
    prm = oracle_params(stack, l)
    k = stack.sh.k
    logits = host(b.logits).astype(np.float64)
    rows = np.arange(h0.shape[0]) if sample is None else sample
    if rcep and K_fixed is not None:
        K = int(K_fixed)
        ref_idx, _ = oracle.prefix_route(logits, K, k)
        np.testing.assert_array_equal(host(b.idx), ref_idx)
        ref = oracle.moe_layer_rcep(h0[rows], prm["w_r"], prm["bias"], prm["w_gate_up"], prm["w_down"],
                                    k, p, logits=logits[rows], K_override=[K])
    elif rcep:
        idx_full, w_full = oracle.full_pool_route(logits, k)
        np.testing.assert_array_equal(host(b.idx_full), idx_full)
        mass = oracle.activated_mass(idx_full, w_full, stack.sh.E)
        K_ref = oracle.prefix_length(mass, p, k)
        K = int(host(stack.K_trace)[l, 0])
        assert K == K_ref or near_tie(mass, p, K_ref), (l, K, K_ref)
        ref_idx, _ = oracle.prefix_route(logits, K, k)
        np.testing.assert_array_equal(host(b.idx), ref_idx)
        ref = oracle.moe_layer_rcep(h0[rows], prm["w_r"], prm["bias"], prm["w_gate_up"], prm["w_down"],
                                    k, p, logits=logits[rows], K_override=[K])
    else:
        ref_idx, _ = oracle.full_pool_route(logits, k)
        np.testing.assert_array_equal(host(b.idx), ref_idx)
        ref = oracle.moe_layer_dense(h0[rows], prm["w_r"], prm["bias"], prm["w_gate_up"],
                                     prm["w_down"], k, logits=logits[rows])
        K = None
    out = host(b.out)[rows]
    assert rel_inf(out, ref["out"]) <= TOL[dt], l
    assert row_rel(out, ref["out"]) <= TOL[dt], l
    # residual update, rounded once
    h1 = host(dst)[rows]
    exp = h0[rows] + ref["out"]
    bound = TOL[dt] * np.abs(ref["out"]).max() + EPS[dt] * np.abs(exp)
    assert (np.abs(h1 - exp) <= bound).all(), l
    return dst, K


def test_tiny_stack_f32_teacher_forced_and_free_running():
    """6 fp32 layers, 384 visual + 128 text rows, exit at layer 3: every
    layer teacher-forced against the oracle; the stack's own forward gives
    the same rows bit for bit; and the oracle's free-running stack agrees
    with it within the fp32 tolerance."""
    wl = I.WORKLOADS["tiny_stack_f32"]
    sh = wl.shape
    st = MoEStack(wl)
    for l in range(st.L):
        check_order(st, l)
    x_np = I.tokens(sh, wl.T, seed=wl.seed)
    x = torch.from_numpy(x_np).cuda()
    h = x
    Ks = []
    for l in range(st.L):
        if l == wl.exit_layer:
            ht = torch.empty((wl.T - wl.n_visual, sh.d), dtype=torch.float32, device="cuda")
            abi.drop_visual_block(h, 0, wl.n_visual, ht)
            np.testing.assert_array_equal(host(ht), host(h)[wl.n_visual:])
            h = ht
        h, K = check_layer(st, l, h, l >= wl.exit_layer, wl.p, "f32")
        Ks.append(K)
    final = host(h)
    out = st.forward(x, wl.n_visual, wl.p, wl.exit_layer)
    np.testing.assert_array_equal(host(out), final)
    np.testing.assert_array_equal(host(st.K_trace)[wl.exit_layer:, 0], Ks[wl.exit_layer:])
    np.testing.assert_array_equal(host(x), x_np)  # the input rows are not modified
    ref, Kref = oracle.moe_stack(x_np, [oracle_params(st, l) for l in range(st.L)], sh.k, wl.p,
                                 exit_layer=wl.exit_layer, v0=0, v1=wl.n_visual)
    assert [int(K[0]) for K in Kref[wl.exit_layer:]] == Ks[wl.exit_layer:]
    assert rel_inf(final, ref) <= TOL["f32"]


@pytest.mark.parametrize("mode,K_fixed", [("dense", None), ("fixed", 5), ("fixed", 2), ("fixed", 16)])
def test_tiny_stack_ablation_modes(mode, K_fixed):
    """The component-ablation modes of the stack (Table 2): the visual exit
    alone (every expert after the exit) and the exit with a fixed prefix
    instead of Eq. 12 (K = 5, K = k = 2, K = E = 16).  Every layer
    teacher-forced against the oracle; the stack's own forward gives the
    layer-by-layer rows bit for bit; the oracle's free-running stack in the
    same mode agrees within the fp32 tolerance."""
    wl = I.WORKLOADS["tiny_stack_f32"]
    sh = wl.shape
    st = MoEStack(wl)
    x_np = I.tokens(sh, wl.T, seed=wl.seed)
    x = torch.from_numpy(x_np).cuda()
    h = x
    for l in range(st.L):
        if l == wl.exit_layer:
            ht = torch.empty((wl.T - wl.n_visual, sh.d), dtype=torch.float32, device="cuda")
            abi.drop_visual_block(h, 0, wl.n_visual, ht)
            h = ht
        after = l >= wl.exit_layer
        h, K = check_layer(st, l, h, after and mode == "fixed", wl.p, "f32",
                           K_fixed=K_fixed if after else None)
        if after and mode == "fixed":
            assert K == K_fixed
    final = host(h)
    out = st.forward(x, wl.n_visual, wl.p, wl.exit_layer, after_exit=mode, K_fixed=K_fixed)
    np.testing.assert_array_equal(host(out), final)
    ref, Kref = oracle.moe_stack(x_np, [oracle_params(st, l) for l in range(st.L)], sh.k, wl.p,
                                 exit_layer=wl.exit_layer, v0=0, v1=wl.n_visual, after_exit=mode,
                                 K_fixed=K_fixed)
    if mode == "fixed":
        assert all(int(K[0]) == K_fixed for K in Kref[wl.exit_layer:])
    else:
        assert all(K is None for K in Kref)
    assert rel_inf(final, ref) <= TOL["f32"]
    with pytest.raises(ValueError):
        st.forward(x, wl.n_visual, wl.p, wl.exit_layer, after_exit="fixed", K_fixed=sh.k - 1)


def test_tiny_stack_gated_exit():
    """SAVB gate at candidate layers 1..5 of the tiny stack: every evaluated
    p_exit matches the oracle's gate on the GPU's text rows entering that
    layer (teacher-forced), the stack exits at the first candidate whose
    p_exit reaches theta, and the result equals the fixed-exit stack at
    that layer bit for bit."""
    wl = I.WORKLOADS["tiny_stack_f32"]
    sh = wl.shape
    st = MoEStack(wl)
    x_np = I.tokens(sh, wl.T, seed=wl.seed)
    x = torch.from_numpy(x_np).cuda()
    gp = {l: I.gate_params(sh.d, seed=wl.seed, layer=l, std=0.1) for l in range(1, st.L)}
    gates = {l: {k: torch.from_numpy(v).cuda() for k, v in g.items()} for l, g in gp.items()}
    # pass 1: theta above 1 never exits; it records p_exit at every candidate
    _, ex0, trace0 = st.forward_gated(x, wl.n_visual, wl.p, gates, 2.0)
    assert ex0 is None and [l for l, _ in trace0] == list(range(1, st.L))
    # the rows entering each candidate layer, from the ungated (all dense) run
    h = x
    for l in range(st.L):
        if l in gp:
            text = host(h)[wl.n_visual:]
            p_ref, _, _, _ = oracle.savb_gate(text, gp[l]["w1"], gp[l]["b1"], gp[l]["w2"], gp[l]["b2"], 0.5)
            assert abs(dict(trace0)[l] - p_ref) <= 1e-5
        dst = torch.empty_like(h)
        st.layer_forward(l, h, dst, False, wl.p)
        h = dst
    # pass 2: theta = the largest p_exit seen -> exit at its first candidate
    ps = [pv for _, pv in trace0]
    theta = max(ps)
    expect = trace0[ps.index(theta)][0]
    out, ex, trace = st.forward_gated(x, wl.n_visual, wl.p, gates, theta)
    assert ex == expect and trace[-1][0] == expect
    got = host(out).copy()  # the stack reuses its buffers
    ref = st.forward(x, wl.n_visual, wl.p, expect)
    np.testing.assert_array_equal(got, host(ref))


@pytest.fixture(scope="module")
def stack48():
    wl = I.WORKLOADS["qwen3vl_stack48_8192"]
    return MoEStack(wl)


def test_stack48_prefill(stack48):
    """48 layers over 7680 visual + 512 text rows, exit at 20 (the bench's
    prefill): teacher-forced against the oracle at dense layers 0, 5, 10, 15
    and 19 (on sampled rows) and at every RCEP layer 20-47 (every row, K
    exact unless a declared near-tie), K of every RCEP layer in the expected
    window, and the stack's forward equals the layer-by-layer run bitwise."""
    st = stack48
    wl = st.wl
    sh = wl.shape
    checked = {0, 5, 10, 15, 19} | set(range(wl.exit_layer, st.L))
    for l in (0, 19, 20, 47):
        check_order(st, l)
    x_np = I.tokens(sh, wl.T, seed=wl.seed)
    x = to_device(x_np, torch.bfloat16)
    rng = np.random.default_rng(5)
    sample = np.unique(np.concatenate([[0, wl.n_visual - 1, wl.n_visual, wl.T - 1],
                                       rng.choice(wl.T, 44, replace=False)]))
    h = x.clone()
    for l in range(st.L):
        if l == wl.exit_layer:
            ht = torch.empty((wl.T - wl.n_visual, sh.d), dtype=torch.bfloat16, device="cuda")
            abi.drop_visual_block(h, 0, wl.n_visual, ht)
            h = ht
        rcep = l >= wl.exit_layer
        if l in checked:
            h, _ = check_layer(st, l, h, rcep, wl.p, "bf16", sample=None if rcep else sample)
        else:
            dst = torch.empty_like(h)
            st.layer_forward(l, h, dst, rcep, wl.p)
            h = dst
    final = host(h)
    Ks = host(st.K_trace)[wl.exit_layer:, 0]
    print("K per RCEP layer", Ks.tolist())
    # the prefix prunes in every RCEP layer (the single layer at this shape
    # keeps 70-90 of 128 experts; the stack's hidden rows drift from the
    # calibration rows' layer by layer, so the window is wider)
    assert ((Ks >= 60) & (Ks <= 115)).all(), Ks
    out = st.forward(x, wl.n_visual, wl.p, wl.exit_layer)
    np.testing.assert_array_equal(host(out), final)
    np.testing.assert_array_equal(host(st.K_trace)[wl.exit_layer:, 0], Ks)
    assert np.isfinite(final).all()


def test_decode64_graph(stack48):
    """64 decode tokens through the same 48 layers, RCEP in every layer
    (p = 0.85): every layer teacher-forced against the oracle (indices, K
    and the layer output); the HIP graph of the step
    replays the eager result bit for bit, three times, with eager work and
    host synchronisation between replays."""
    st = stack48
    wl = I.WORKLOADS["qwen3vl_decode64"]
    sh = wl.shape
    x_np = I.tokens(sh, wl.T, seed=wl.seed, stream="decode")
    x = to_device(x_np, torch.bfloat16)
    h = x.clone()
    for l in range(st.L):
        h, _ = check_layer(st, l, h, True, wl.p, "bf16")
    eager = host(h)
    Ks = host(st.K_trace)[:, 0].copy()
    assert ((Ks >= sh.k) & (Ks <= sh.E)).all()
    out = st.forward(x, 0, wl.p, exit_layer=0)
    np.testing.assert_array_equal(host(out), eager)
    assert st.chainable()
    np.testing.assert_array_equal(host(st.forward_decode(x, wl.p)), eager)
    g, gout = st.capture_decode(x, wl.p)
    other = to_device(I.tokens(sh, wl.T, seed=wl.seed + 1, stream="decode"), torch.bfloat16)
    for rep in range(3):
        st.K_trace.zero_()
        gout.zero_()
        g.replay()
        torch.cuda.synchronize()
        np.testing.assert_array_equal(host(gout), eager)
        np.testing.assert_array_equal(host(st.K_trace)[:, 0], Ks)
        st.forward(other, 0, wl.p, exit_layer=0)  # eager work between replays
        torch.cuda.synchronize()
