"""Layer parity: the composed dense and RCEP spans (Algorithm 2) on the GPU
against the oracle, at the workload sizes, in the launch configuration the
bench times (packed bf16 expert weights, the same buffers and calls).

Protocol (teacher-forced where floating point decides an integer): the
oracle routes from the GPU's float32 logits widened to float64, so expert
indices, K and the Mean-Mass order are compared bit for bit; outputs are
compared with ||y - y_ref||_inf / ||y_ref||_inf <= 2e-2 (bf16) or 1e-4
(fp32), and per row with the floor of 1e-3 rms.  At 4096 rows the oracle
evaluates a seeded sample of tokens; the dense layer's routing is per token,
so a sample needs no other rows.
"""

from types import SimpleNamespace

import numpy as np
import pytest
import torch

import oracle
from _util import ensure_built, rel_inf, row_rel

pytestmark = pytest.mark.gpu

from paper_2609_38823_amd import abi  # noqa: E402
from paper_2609_38823_amd import inputs as I  # noqa: E402
from paper_2609_38823_amd.layer import MoELayer, apply_order, calibrate_order_router  # noqa: E402

TOL = {"f32": 1e-4, "bf16": 2e-2}
TDT = {"f32": torch.float32, "bf16": torch.bfloat16}


@pytest.fixture(scope="module", autouse=True)
def _lib():
    ensure_built()
    torch.cuda.init()


def host(t):
    torch.cuda.synchronize()
    return (t.float() if t.dtype == torch.bfloat16 else t).cpu().numpy()


def near_tie(mass, p, K, k, rel=1e-9):
    """True if K is decided by a float64 near-tie: c_{K_hat} or c_{K_hat - 1}
    lies within rel * tot of p * tot (then either K is a valid reading)."""
    c = np.cumsum(np.asarray(mass, np.float64))
    tot, thr = c[-1], p * c[-1]
    k_hat = np.searchsorted(c >= thr, True) + 1
    m = min(abs(c[k_hat - 1] - thr), abs(thr - c[k_hat - 2]) if k_hat >= 2 else np.inf)
    return m < rel * tot


def calibrated_layer(wl, calib_x):
    """Mean-Mass order from the GPU's full-pool routing of the calibration
    rows, checked against the oracle's order of that same routing, then the
    physical reorder and the device layer."""
    sh = wl.shape
    prm = I.layer_params(sh, seed=wl.seed)
    xc = torch.from_numpy(calib_x).cuda().to(TDT[sh.dtype])
    order = calibrate_order_router(xc, prm["w_r"], prm["bias"], sh.k)
    # teacher-forced order: the oracle's Eq. 8-9 on the GPU's routing
    T, E = calib_x.shape[0], sh.E
    logits = torch.empty((T, E), dtype=torch.float32, device="cuda")
    idx = torch.empty((T, sh.k), dtype=torch.int32, device="cuda")
    w = torch.empty((T, sh.k), dtype=torch.float32, device="cuda")
    ws = torch.empty(abi.moe_workspace_size(T, E, sh.k, sh.d, 1, 1), dtype=torch.uint8, device="cuda")
    abi.moe_route(xc, torch.from_numpy(prm["w_r"]).cuda(),
                  torch.from_numpy(prm["bias"]).cuda() if prm["bias"] is not None else None,
                  sh.k, logits, idx, w, ws=ws)
    M = oracle.routed_mass(host(idx), host(w).astype(np.float64), E)
    np.testing.assert_array_equal(order, oracle.mean_mass_order(M[None, :])[0])
    rp = apply_order(prm, order)
    return rp, MoELayer(rp, sh.k, sh.dtype)


@pytest.fixture(scope="module")
def qwen():
    wl = I.WORKLOADS["qwen3vl_dense_4096"]
    x = I.tokens(wl.shape, wl.T, seed=wl.seed)
    rp, layer = calibrated_layer(wl, x[wl.n_visual:])
    return wl, x, rp, layer


def check_dense(layer, rp, x_np, xd, k, dt, sample=None):
    b = layer.forward_dense(xd)
    logits = host(b.logits).astype(np.float64)
    ref_idx, _ = oracle.full_pool_route(logits, k)
    np.testing.assert_array_equal(host(b.idx), ref_idx)  # every token
    counts = host(b.counts)
    assert counts.sum() == x_np.shape[0] * k
    np.testing.assert_array_equal(host(b.offsets), np.concatenate([[0], np.cumsum(counts)]))
    rows = np.arange(x_np.shape[0]) if sample is None else sample
    ref = oracle.moe_layer_dense(x_np[rows], rp["w_r"], rp["bias"], rp["w_gate_up"], rp["w_down"], k,
                                 logits=logits[rows])
    out = host(b.out)[rows]
    assert rel_inf(out, ref["out"]) <= TOL[dt]
    assert row_rel(out, ref["out"]) <= TOL[dt]
    return b


def check_rcep(layer, rp, x_np, xd, k, p, dt, sample=None):
    b = layer.forward_rcep(xd, p)
    logits = host(b.logits).astype(np.float64)
    # K from the oracle's Eqs. 10-12 on the GPU logits
    idx_full, w_full = oracle.full_pool_route(logits, k)
    np.testing.assert_array_equal(host(b.idx_full), idx_full)
    mass = oracle.activated_mass(idx_full, w_full, layer.E)
    K_ref = oracle.prefix_length(mass, p, k)
    K = int(host(b.K)[0])
    assert K == K_ref or near_tie(mass, p, K_ref, k), (K, K_ref)
    ref_idx, _ = oracle.prefix_route(logits, K, k)
    gi = host(b.idx)
    np.testing.assert_array_equal(gi, ref_idx)
    assert gi.max() < K
    counts = host(b.counts)
    assert (counts[K:] == 0).all() and counts.sum() == x_np.shape[0] * k
    rows = np.arange(x_np.shape[0]) if sample is None else sample
    ref = oracle.moe_layer_rcep(x_np[rows], rp["w_r"], rp["bias"], rp["w_gate_up"], rp["w_down"], k, p,
                                logits=logits[rows], K_override=[K])
    out = host(b.out)[rows]
    assert rel_inf(out, ref["out"]) <= TOL[dt]
    assert row_rel(out, ref["out"]) <= TOL[dt]
    return b, K


def test_tiny_fp32_layer_end_to_end():
    """Tiny fp32 layer: order calibrated on the text rows, dense span over
    all 512 rows, SAVB drop of rows 0-383, RCEP span over the text rows."""
    wl = I.WORKLOADS["tiny_f32"]
    sh = wl.shape
    x = I.tokens(sh, wl.T, seed=wl.seed)
    rp, layer = calibrated_layer(wl, x[wl.n_visual:])
    xd = torch.from_numpy(x).cuda()
    check_dense(layer, rp, x, xd, sh.k, sh.dtype)
    h = torch.empty((wl.T - wl.n_visual, sh.d), dtype=torch.float32, device="cuda")
    abi.drop_visual_block(xd, 0, wl.n_visual, h)
    np.testing.assert_array_equal(host(h), x[wl.n_visual:])
    check_rcep(layer, rp, x[wl.n_visual:], h, sh.k, wl.p, sh.dtype)


def test_qwen_dense_4096_sampled(qwen):
    """Dense span over 3584 visual + 512 text rows (the bench's dense call)."""
    wl, x, rp, layer = qwen
    assert layer.packed
    rng = np.random.default_rng(11)
    sample = np.unique(np.concatenate([[0, wl.n_visual - 1, wl.n_visual, wl.T - 1],
                                       rng.choice(wl.T, 60, replace=False)]))
    xd = torch.from_numpy(x).cuda().to(torch.bfloat16)
    b = check_dense(layer, rp, x, xd, wl.shape.k, "bf16", sample=sample)
    assert int((host(b.counts) > 0).sum()) == wl.shape.E


def test_qwen_rcep_512(qwen):
    """RCEP span over the 512 text rows after the visual exit (p = 0.9): K in
    the configured window, prefix re-route, experts [0, K) only."""
    wl, x, rp, layer = qwen
    text = x[wl.n_visual:]
    xd = torch.from_numpy(text).cuda().to(torch.bfloat16)
    rng = np.random.default_rng(12)
    sample = np.unique(np.concatenate([[0, 511], rng.choice(512, 126, replace=False)]))
    _, K = check_rcep(layer, rp, text, xd, wl.shape.k, I.WORKLOADS["qwen3vl_rcep_512"].p, "bf16",
                      sample=sample)
    assert 70 <= K <= 90, K


def test_rcep_with_full_support_and_p_one_equals_dense(qwen):
    """p = 1 keeps every expert with positive mass; when all 128 have mass
    the prefix is the full pool and the RCEP span must reproduce the dense
    span bit for bit (same routing, same kernels)."""
    wl, x, rp, layer = qwen
    xd = torch.from_numpy(x[wl.n_visual:]).cuda().to(torch.bfloat16)
    bd = layer.forward_dense(xd)
    out_d = host(bd.out).copy()
    br = layer.forward_rcep(xd, 1.0)
    if int((host(br.mass)[0] > 0).sum()) == wl.shape.E:
        assert int(host(br.K)[0]) == wl.shape.E
        np.testing.assert_array_equal(host(br.out), out_d)


def test_rcep_is_deterministic(qwen):
    """Two runs of the RCEP span give bitwise identical results."""
    wl, x, rp, layer = qwen
    xd = torch.from_numpy(x[wl.n_visual:]).cuda().to(torch.bfloat16)
    b1 = layer.forward_rcep(xd, 0.9)
    r1 = [host(t).copy() for t in (b1.logits, b1.mass, b1.K, b1.idx, b1.w, b1.out)]
    b2 = layer.forward_rcep(xd, 0.9)
    r2 = [host(t) for t in (b2.logits, b2.mass, b2.K, b2.idx, b2.w, b2.out)]
    for a, b in zip(r1, r2):
        np.testing.assert_array_equal(a, b)


def test_decode_64_layer():
    """Decode regime: 64 single text tokens, p = 0.85, order calibrated on a
    separate 512-row calibration set of the layer."""
    wl = I.WORKLOADS["qwen3vl_decode64"]
    sh = wl.shape
    calib = I.tokens(sh, 512, seed=wl.seed, stream="calib")
    rp, layer = calibrated_layer(wl, calib)
    x = I.tokens(sh, wl.T, seed=wl.seed, stream="decode")
    xd = torch.from_numpy(x).cuda().to(torch.bfloat16)
    check_rcep(layer, rp, x, xd, sh.k, wl.p, "bf16")


def test_dense_equivalent_executor_matches_sparse(qwen):
    """The paper's dense-equivalent execution (App. A.3): every text token
    through all K retained experts with the sparse routing weights applied
    afterwards (zero for unselected experts) gives the sparse layer's
    output; each retained expert gets every token."""
    wl, x, rp, layer = qwen
    sh = wl.shape
    text = x[wl.n_visual:]
    T, E = text.shape[0], sh.E
    xd = torch.from_numpy(text).cuda().to(torch.bfloat16)
    b = layer.forward_rcep(xd, 0.9)
    out_sparse = host(b.out).copy()
    K = int(host(b.K)[0])
    idx_d = torch.empty((T, E), dtype=torch.int32, device="cuda")
    w_d = torch.empty((T, E), dtype=torch.float32, device="cuda")
    abi.moe_expand_dense_routing(b.idx, b.w, E, idx_d, w_d, K_dev=b.K)
    gi, gw = host(idx_d), host(w_d)
    slots = np.arange(E)[None, :].repeat(T, axis=0)
    np.testing.assert_array_equal(gi, np.where(slots < K, slots, -1))
    ref_w = np.zeros((T, E), np.float32)
    np.put_along_axis(ref_w, host(b.idx).astype(np.int64), host(b.w), axis=1)
    np.testing.assert_array_equal(gw, ref_w)
    from paper_2609_38823_amd.layer import Buffers
    bd = Buffers(T, sh.d, E, sh.m, E, torch.bfloat16)
    abi.moe_dispatch(idx_d, E, xd, bd.counts, bd.offsets, bd.src_of_row, bd.row_of_slot, bd.x_perm, bd.ws)
    counts = host(bd.counts)
    assert (counts[:K] == T).all() and (counts[K:] == 0).all()
    abi.moe_expert_ffn_packed(bd.x_perm, bd.offsets, layer.w_gate_up, layer.w_down, bd.y_perm, bd.ws,
                              K_dev=b.K)
    abi.moe_combine(bd.y_perm, bd.row_of_slot, w_d, bd.out)
    out_dense = host(bd.out)
    assert rel_inf(out_dense, out_sparse) <= 2e-2
    # the same eight products per element, summed in another order: within
    # a few bf16 units of the sparse result
    assert np.abs(out_dense - out_sparse).max() <= 4 * 2.0 ** -8 * np.abs(out_sparse).max()
    # and against the oracle's RCEP layer at the GPU's K (teacher-forced on
    # the GPU's logits), element by element over every text row
    logits = host(b.logits).astype(np.float64)
    ref = oracle.moe_layer_rcep(text, rp["w_r"], rp["bias"], rp["w_gate_up"], rp["w_down"], sh.k, 0.9,
                                logits=logits, K_override=[K])
    np.testing.assert_array_equal(host(b.idx), ref["idx"])
    assert rel_inf(out_dense, ref["out"]) <= TOL["bf16"]
    assert row_rel(out_dense, ref["out"]) <= TOL["bf16"]


@pytest.mark.parametrize("K", [8, 50, 85, 128])
def test_fixed_prefix_layer(qwen, K):
    """The fixed-prefix variant of the component ablation (Table 2: a prefix
    of 50 instead of Eq. 12; the keep ratios of the order study): the split
    router's logits over all 128 experts, Top-k inside [0, K), the expert FFN
    over experts [0, K) only.  Indices bit-exact and outputs within 2e-2 of
    the oracle's layer at that K on the GPU's logits, every text row."""
    wl, x, rp, layer = qwen
    sh = wl.shape
    text = x[wl.n_visual:]
    xd = torch.from_numpy(text).cuda().to(torch.bfloat16)
    assert layer.w_r_packed is not None  # the bf16 split router path (moe_route_packed with K_dev)
    b = layer.forward_prefix(xd, K)
    logits = host(b.logits).astype(np.float64)
    ref = oracle.moe_layer_rcep(text, rp["w_r"], rp["bias"], rp["w_gate_up"], rp["w_down"], sh.k, 0.9,
                                logits=logits, K_override=[K])
    gi = host(b.idx)
    np.testing.assert_array_equal(gi, ref["idx"])
    assert gi.max() < K
    counts = host(b.counts)
    np.testing.assert_array_equal(counts, ref["counts"])
    assert (counts[K:] == 0).all()
    np.testing.assert_array_equal(host(b.row_of_slot), ref["row_of_slot"])
    np.testing.assert_allclose(host(b.w), ref["w"], rtol=1e-5, atol=1e-7)
    out = host(b.out)
    assert rel_inf(out, ref["out"]) <= TOL["bf16"]
    assert row_rel(out, ref["out"]) <= TOL["bf16"]


def test_fixed_prefix_below_k(qwen):
    """Eq. 12 gives K >= k, so a host prefix below k is rejected; a device
    value below k is raised to k by the route and by the gathering expert
    FFN alike (bitwise the result at K = k)."""
    wl, x, rp, layer = qwen
    text = x[wl.n_visual:]
    xd = torch.from_numpy(text).cuda().to(torch.bfloat16)
    with pytest.raises(ValueError):
        layer.forward_prefix(xd, wl.shape.k - 1)
    with pytest.raises(ValueError):
        layer.forward_prefix(xd, wl.shape.E + 1)
    ref = host(layer.forward_prefix(xd, wl.shape.k).out).copy()
    K_dev = torch.full((4,), 3, dtype=torch.int32, device="cuda")[:1]
    got = host(layer.forward_prefix(xd, K_dev).out)
    np.testing.assert_array_equal(got, ref)


def _sweep_cases():
    """Seeded random layer shapes on both expert-FFN paths: bf16 with packed
    weights (d, m multiples of 256) or row-major weights (m a multiple of 128
    only), float32 with any d and m; routers on the split-weight, float32
    MFMA and scalar paths by E and d."""
    rng = np.random.default_rng(2609)
    cases = []
    for i in range(8):
        E = int(rng.choice([4, 32, 64, 96, 160, 256]))
        cases.append(("bf16", int(rng.choice([256, 512, 768])), E, int(rng.choice([128, 256, 384, 512])),
                      int(rng.integers(1, min(8, E) + 1)), int(rng.choice([1, 37, 300, 1000])),
                      float(rng.choice([0.5, 0.8, 0.9, 1.0])), bool(rng.integers(0, 2)), i))
    for i in range(6):
        E = int(rng.choice([3, 16, 50, 128]))
        cases.append(("f32", int(rng.choice([24, 64, 200, 256])), E, int(rng.choice([12, 40, 96])),
                      int(rng.integers(1, min(8, E) + 1)), int(rng.choice([1, 37, 300, 700])),
                      float(rng.choice([0.5, 0.8, 0.9, 1.0])), bool(rng.integers(0, 2)), 100 + i))
    return cases


@pytest.mark.parametrize("dt,d,E,m,k,T,p,bias,seed", _sweep_cases())
def test_layer_shape_sweep(dt, d, E, m, k, T, p, bias, seed):
    """Dense and RCEP spans on random shapes against the oracle (same
    protocol as the workload tests)."""
    sh = I.LayerShape(d=d, E=E, m=m, k=k, dtype=dt, zipf_alpha=0.35 if bias else None)
    wl = SimpleNamespace(shape=sh, seed=seed)
    x = I.tokens(sh, T, seed=seed)
    print(f"sweep case {dt} d={d} E={E} m={m} k={k} T={T} p={p} bias={bias}", flush=True)
    rp, layer = calibrated_layer(wl, x)
    xd = torch.from_numpy(x).cuda().to(TDT[dt])
    check_dense(layer, rp, x, xd, k, dt)
    check_rcep(layer, rp, x, xd, k, p, dt)
    if layer.packed and layer.w_r_packed is not None:
        # with the residual the layer is one call (moe_rcep_layer); the
        # separate calls (forced by a stage marker) give the same bits
        outs = []
        for mark in (None, lambda: None):
            out = torch.empty_like(xd)
            b = layer.forward_rcep(xd, p, residual=xd, out=out, mark=mark)
            outs.append((out, b.K.clone(), b.idx.clone()))
        torch.cuda.synchronize()
        assert torch.equal(outs[0][0].view(torch.int16), outs[1][0].view(torch.int16))
        assert torch.equal(outs[0][1], outs[1][1]) and torch.equal(outs[0][2], outs[1][2])


@pytest.mark.parametrize("sizes", [[1] * 64, [1, 7, 0, 20, 36]])
def test_rcep_per_sequence_segments(qwen, sizes):
    """One invocation per sequence (Eq. 11's token set is the segment): K per
    segment from the oracle on the GPU's logits, each token re-routed inside
    its own segment's prefix, the expert FFN over the experts below the
    largest K, and the output against the oracle (64 decode tokens, one
    segment per token or ragged segments with an empty one)."""
    wl, _, rp, layer = qwen
    sh = wl.shape
    x_np = I.tokens(sh, 64, seed=5)
    xd = torch.from_numpy(x_np).cuda().to(torch.bfloat16)
    so = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    seg = torch.from_numpy(so).cuda()
    p = 0.85
    b = layer.forward_rcep(xd, p, seg_offsets=seg)
    logits = host(b.logits).astype(np.float64)
    idx_full, w_full = oracle.full_pool_route(logits, sh.k)
    np.testing.assert_array_equal(host(b.idx_full), idx_full)
    K = host(b.K).astype(np.int64)
    K_ref = np.array([oracle.prefix_length(oracle.activated_mass(idx_full[lo:hi], w_full[lo:hi], sh.E),
                                           p, sh.k) for lo, hi in zip(so[:-1], so[1:])])
    for s, (lo, hi) in enumerate(zip(so[:-1], so[1:])):
        mass = oracle.activated_mass(idx_full[lo:hi], w_full[lo:hi], sh.E)
        assert K[s] == K_ref[s] or near_tie(mass, p, K_ref[s], sh.k), (s, K[s], K_ref[s])
    ref = oracle.moe_layer_rcep(x_np, rp["w_r"], rp["bias"], rp["w_gate_up"], rp["w_down"], sh.k, p,
                                seg_offsets=so, logits=logits, K_override=K)
    gi = host(b.idx)
    np.testing.assert_array_equal(gi, ref["idx"])
    for s, (lo, hi) in enumerate(zip(so[:-1], so[1:])):
        assert (gi[lo:hi] < K[s]).all()
    counts = host(b.counts)
    assert counts.sum() == 64 * sh.k and (counts[K.max():] == 0).all()
    out = host(b.out)
    assert rel_inf(out, ref["out"]) <= TOL["bf16"]
    assert row_rel(out, ref["out"]) <= TOL["bf16"]
