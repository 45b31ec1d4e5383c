"""Stage parity: every C-ABI entry point against the oracle on identical
seeded inputs (GPU).

Integer results (indices, counts, offsets, permutations, K, order) must be
bit-exact; the row copies (dispatch gather, visual drop) bitwise; floating
outputs within the stated tolerance:
  logits   |a - a_ref| <= gamma_{d+2} (sum_j |x_j W_je| + |b_e|)
  weights  relative 1e-5
  FFN and combine outputs  ||y - y_ref||_inf / ||y_ref||_inf <= 2e-2 (bf16),
           1e-4 (fp32), and the same bound per row (floor 1e-3 rms)
"""

import numpy as np
import pytest
import torch

import oracle
from _util import ensure_built, gamma, rel_inf, row_rel

pytestmark = pytest.mark.gpu

from paper_2609_38823_amd import abi  # noqa: E402
from paper_2609_38823_amd import inputs as I  # noqa: E402
from paper_2609_38823_amd.layer import to_device  # noqa: E402

TDT = {"f32": torch.float32, "bf16": torch.bfloat16}
TOL = {"f32": 1e-4, "bf16": 2e-2}


@pytest.fixture(scope="module", autouse=True)
def _lib():
    ensure_built()
    torch.cuda.init()


def dev(a, dtype=None):
    a = np.ascontiguousarray(a)
    t = torch.from_numpy(a).cuda()
    return t.to(dtype) if dtype is not None else t


def host(t):
    torch.cuda.synchronize()
    if t.dtype == torch.bfloat16:
        t = t.float()
    return t.cpu().numpy()


def host_bits(t):
    """uint16 bit patterns of a bf16 device tensor."""
    torch.cuda.synchronize()
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def i32(shape):
    return torch.full(shape, -7, dtype=torch.int32, device="cuda")


def f32(shape):
    return torch.full(shape, float("nan"), dtype=torch.float32, device="cuda")


def assert_ffn_ran_all(ws):
    """The last expert FFN call on ws evaluated every item of its plan and
    no down item gave up waiting for its h (moe_ffn_status)."""
    st = torch.full((4,), -1, dtype=torch.int32, device="cuda")
    abi.moe_ffn_status(ws, st)
    gave_up, done, planned, path = (int(v) for v in host(st))
    assert path in (abi.FFN_PATH_PERSISTENT, abi.FFN_PATH_TWO_LAUNCH, abi.FFN_PATH_ROW_MAJOR,
                    abi.FFN_PATH_F32), path
    assert gave_up == 0
    assert done == planned
    if path != abi.FFN_PATH_PERSISTENT:
        assert done == planned == 0
    return path, planned


def ws_for(T, E, k, d, m=1, n_seg=1):
    """Workspace for any entry point at these sizes (moe_workspace_size)."""
    return torch.empty(abi.moe_workspace_size(max(T, 1), E, k, d, m, n_seg), dtype=torch.uint8,
                       device="cuda")


# ---------------------------------------------------------------------------
# drop_visual_block (Sec. 3.2, Algorithm 2): bitwise row compaction
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("dt", ["f32", "bf16"])
@pytest.mark.parametrize("S,d,v0,v1", [(512, 256, 0, 384), (8192, 2048, 0, 7680), (37, 24, 5, 17),
                                       (10, 8, 0, 10), (10, 8, 3, 3), (1, 8, 0, 0), (100, 6, 90, 100),
                                       (65, 2, 1, 64)])
def test_drop_visual_block_bitwise(dt, S, d, v0, v1):
    h = I.synthetic_rows(S, d, dt, seed=S + d)
    hd = dev(h, TDT[dt])
    out = torch.full((S - (v1 - v0), d), -1.0, dtype=TDT[dt], device="cuda")
    abi.drop_visual_block(hd, v0, v1, out)
    ref = oracle.drop_visual_block(h, v0, v1)
    got = host(out)
    assert got.shape == ref.shape
    np.testing.assert_array_equal(got.view(np.uint32), ref.view(np.uint32))


# ---------------------------------------------------------------------------
# moe_route, logits-input mode: Top-k and weights on given logits
# ---------------------------------------------------------------------------
# T >= 4096 takes the four-tokens-per-wavefront kernel (8 or 16 values per
# lane; k > 16 uses the second slot of every lane)
ROUTE_CASES = [(1, 16, 2), (37, 16, 2), (5, 7, 7), (129, 64, 1), (512, 128, 8), (4095, 128, 8),
               (4096, 128, 8), (300, 1000, 32), (70, 65, 3), (16384, 128, 8), (5000, 200, 20),
               (16390, 200, 20), (16385, 100, 32)]


@pytest.mark.parametrize("ties", [False, True])
@pytest.mark.parametrize("T,E,k", ROUTE_CASES)
def test_topk_on_given_logits(T, E, k, ties):
    a = I.logits_with_ties(T, E, seed=E) if ties else I.synthetic_rows(T, E, "f32", seed=T * E)
    logits = dev(a)
    idx, w = i32((T, k)), f32((T, k))
    abi.moe_route(None, None, None, k, logits, idx, w)
    ref_idx, ref_w = oracle.full_pool_route(a, k)
    np.testing.assert_array_equal(host(idx), ref_idx)
    np.testing.assert_allclose(host(w), ref_w, rtol=1e-5, atol=1e-7)


@pytest.mark.parametrize("T,E,k,segs,Ks", [
    (512, 16, 2, [0, 512], [9]),
    (512, 128, 8, [0, 512], [84]),
    (64, 128, 8, list(range(65)), None),  # one token per segment
    (200, 128, 8, [0, 0, 50, 50, 130, 200], [8, 40, 3, 128, 200]),  # empty segments, clamping
    (33, 10, 4, [0, 33], [4]),  # K == k
    (16390, 256, 17, [0, 8000, 8000, 16390], [100, 5, 256]),  # row kernel, 16 values per lane
    (16384, 128, 8, [0, 16384], [84]),
])
def test_prefix_reroute_on_given_logits(T, E, k, segs, Ks):
    a = I.synthetic_rows(T, E, "f32", seed=7 * T + E)
    n_seg = len(segs) - 1
    if Ks is None:
        Ks = list(np.random.default_rng(0).integers(k, E + 1, size=n_seg))
    idx, w = i32((T, k)), f32((T, k))
    abi.moe_route(None, None, None, k, dev(a), idx, w, seg_offsets=dev(np.array(segs, np.int32)),
                  K_dev=dev(np.array(Ks, np.int32)))
    gi, gw = host(idx), host(w)
    for s in range(n_seg):
        lo, hi = segs[s], segs[s + 1]
        if hi == lo:
            continue
        K = min(max(Ks[s], k), E)  # the documented clamp to [k, E]
        ri, rw = oracle.prefix_route(a[lo:hi], K, k)
        np.testing.assert_array_equal(gi[lo:hi], ri)
        np.testing.assert_allclose(gw[lo:hi], rw, rtol=1e-5, atol=1e-7)


# ---------------------------------------------------------------------------
# moe_route, logits from x: bounded logit error, free-running Top-k
# ---------------------------------------------------------------------------
def logit_bound(x, w_r, bias):
    d = x.shape[1]
    mag = np.abs(x.astype(np.float64)) @ np.abs(w_r.astype(np.float64))
    if bias is not None:
        mag = mag + np.abs(bias.astype(np.float64))[None, :]
    return gamma(d + 2) * mag


def robust_tokens(a_ref, k, delta):
    """Tokens whose Top-k set and slot order cannot change under a logit
    perturbation of at most delta[t]: every gap among the k+1 largest
    logits exceeds 2 delta[t]."""
    srt = -np.sort(-a_ref, axis=1)[:, :k + 1]
    if srt.shape[1] < 2:
        return np.ones(a_ref.shape[0], bool)
    return (-np.diff(srt, axis=1)).min(axis=1) > 2 * delta


ODD_F32 = I.LayerShape(d=40, E=24, m=8, k=3, dtype="f32", zipf_alpha=0.35)
ODD_BF16 = I.LayerShape(d=104, E=200, m=8, k=8, dtype="bf16", zipf_alpha=0.35)
# d-range splits: tiny 512 / 37 -> 2, qwen 4096 -> 1, 512 -> 8, 77, 64 and 1 -> 16;
# the odd shapes take the SIMT kernel
ROUTER_CASES = [("tiny_f32", 512), ("tiny_f32", 37), ("qwen3vl_dense_4096", 4096),
                ("qwen3vl_rcep_512", 512), ("qwen3vl_dense_4096", 77), ("qwen3vl_decode64", 64),
                ("qwen3vl_rcep_512", 1), ("odd_f32", 99), ("odd_bf16", 333)]


@pytest.mark.parametrize("name,T", ROUTER_CASES)
def test_router_logits_and_free_running_topk(name, T):
    if name == "odd_f32":
        wl, sh = I.Workload(name, ODD_F32, T, 0, 0.9), ODD_F32
    elif name == "odd_bf16":
        wl, sh = I.Workload(name, ODD_BF16, T, 0, 0.9), ODD_BF16
    else:
        wl = I.WORKLOADS[name]
        sh = wl.shape
    rp = I.router_params(sh, seed=wl.seed)
    x = I.tokens(sh, T, seed=wl.seed)
    logits, idx, w = f32((T, sh.E)), i32((T, sh.k)), f32((T, sh.k))
    abi.moe_route(dev(x, TDT[sh.dtype]), dev(rp["w_r"]), dev(rp["bias"]) if rp["bias"] is not None else None,
                  sh.k, logits, idx, w, ws=ws_for(T, sh.E, sh.k, sh.d))
    a_ref = oracle.router_logits(x, rp["w_r"], rp["bias"])
    a_gpu = host(logits).astype(np.float64)
    # every logit within the rigorous float32 dot-product error bound
    assert np.all(np.abs(a_gpu - a_ref) <= logit_bound(x, rp["w_r"], rp["bias"]))
    # Top-k is a pure comparison: wherever the measured logit error cannot
    # reorder the k+1 largest logits, the selection must equal the oracle's
    delta = np.abs(a_gpu - a_ref).max(axis=1)
    ok = robust_tokens(a_ref, sh.k, delta)
    ref_idx, ref_w = oracle.full_pool_route(a_ref, sh.k)
    gi = host(idx)
    np.testing.assert_array_equal(gi[ok], ref_idx[ok])
    assert ok.mean() > 0.99
    # the remaining near-tie tokens still pick a valid Top-k: every chosen
    # logit is within 2 delta of the oracle's k-th largest
    kth = -np.sort(-a_ref, axis=1)[:, sh.k - 1]
    chosen = np.take_along_axis(a_ref, gi.astype(np.int64), axis=1)
    assert np.all(chosen >= (kth - 2 * delta)[:, None])
    np.testing.assert_allclose(host(w)[ok], ref_w[ok], rtol=2e-5, atol=1e-6)


# ---------------------------------------------------------------------------
# moe_pack_router / moe_route_packed: three-term bf16 split of W_r on MFMA
# ---------------------------------------------------------------------------
def split3_np(w):
    """W1 = bf16(W), W2 = bf16(W - W1), W3 = bf16(W - W1 - W2) (float32
    differences, exact)."""
    w = np.asarray(w, np.float32)
    w1 = I.round_to_bf16(w)
    r1 = (w - w1).astype(np.float32)
    w2 = I.round_to_bf16(r1)
    w3 = I.round_to_bf16((r1 - w2).astype(np.float32))
    return w1, w2, w3


def pack_router_np(w):
    """The documented layout: element 8 l + j of block ((eb KB + kb) 3 + p)
    is term p of W[16 kb + 8 (l / 32) + j, 32 eb + l % 32]."""
    d, E = w.shape
    KB = d // 16
    l, j = np.arange(64), np.arange(8)
    k_idx = 16 * np.arange(KB)[:, None, None] + 8 * (l // 32)[None, :, None] + j[None, None, :]
    out = np.empty((E // 32, KB, 3, 64, 8), np.float32)
    for p, P in enumerate(split3_np(w)):
        for eb in range(E // 32):
            out[eb, :, p] = P[k_idx, 32 * eb + (l % 32)[None, :, None]]
    return out.reshape(-1)


E96_BF16 = I.LayerShape(d=256, E=96, m=8, k=4, dtype="bf16", zipf_alpha=0.35)  # 3 of 4 waves busy
E256_BF16 = I.LayerShape(d=128, E=256, m=8, k=8, dtype="bf16", zipf_alpha=0.35)
E256_K20 = I.LayerShape(d=128, E=256, m=8, k=20, dtype="bf16", zipf_alpha=0.35)
D64_BF16 = I.LayerShape(d=64, E=32, m=8, k=2, dtype="bf16", zipf_alpha=None)   # one 64-wide stage


# 64-row tiles at 4096 (4 splits) and 8192 (2); 32-row tiles with 8 splits
# below; from 65 536 rows (E <= 128) 128-row tiles over the whole d-range,
# then the four-tokens-per-wavefront Top-k (ragged last tile, idle
# wavefronts, a single 64-wide stage); the small shapes cover idle
# wavefronts and S = 1 with a single stage
@pytest.mark.parametrize("shape,T", [("qwen", 4096), ("qwen", 8192), ("qwen", 512), ("qwen", 77),
                                     ("qwen", 64), ("qwen", 1), ("e96", 333), ("d64", 50),
                                     ("qwen", 65536), ("qwen", 65536 + 77), ("e96", 65536 + 5),
                                     ("d64", 70000)])
def test_route_packed(shape, T):
    sh = {"qwen": I.QWEN3_VL_MOE, "e96": E96_BF16, "d64": D64_BF16}[shape]
    rp = I.router_params(sh, seed=3)
    x = I.tokens(sh, T, seed=T)
    w_r = dev(rp["w_r"])
    wp = torch.empty((3 * sh.d * sh.E,), dtype=torch.bfloat16, device="cuda")
    abi.moe_pack_router(w_r, wp)
    np.testing.assert_array_equal(host_bits(wp), I.bf16_bits(pack_router_np(rp["w_r"])))
    logits, idx, w = f32((T, sh.E)), i32((T, sh.k)), f32((T, sh.k))
    bias = dev(rp["bias"]) if rp["bias"] is not None else None
    abi.moe_route_packed(dev(x, torch.bfloat16), wp, bias, sh.k, logits, idx, w,
                         ws=ws_for(T, sh.E, sh.k, sh.d))
    a_gpu = host(logits).astype(np.float64)
    rows = np.arange(T) if T <= 8192 else np.random.default_rng(1).choice(T, 4096, replace=False)
    a_ref = oracle.router_logits(x[rows], rp["w_r"], rp["bias"])
    a_gpu = a_gpu[rows]
    # bound: 3d exact products accumulated in float32 plus up to 32 split
    # partials and the bias (gamma_{3d+40}), plus the split's own
    # representation error 2^-24 |W| per term (2^-23 with margin)
    mag = np.abs(x[rows].astype(np.float64)) @ np.abs(rp["w_r"].astype(np.float64))
    full = mag + (np.abs(rp["bias"].astype(np.float64))[None, :] if rp["bias"] is not None else 0)
    assert np.all(np.abs(a_gpu - a_ref) <= gamma(3 * sh.d + 40) * full + 2.0 ** -23 * mag)
    delta = np.abs(a_gpu - a_ref).max(axis=1)
    ok = robust_tokens(a_ref, sh.k, delta)
    ref_idx, ref_w = oracle.full_pool_route(a_ref, sh.k)
    gi = host(idx)[rows]
    np.testing.assert_array_equal(gi[ok], ref_idx[ok])
    assert ok.mean() > 0.99
    # teacher-forced: the Top-k of the GPU's own logits is exact
    tf_idx, tf_w = oracle.full_pool_route(a_gpu, sh.k)
    np.testing.assert_array_equal(gi, tf_idx)
    np.testing.assert_allclose(host(w)[rows], tf_w, rtol=2e-5, atol=1e-6)


@pytest.mark.parametrize("T", [65536 + 300, 4096])
def test_route_packed_prefix_segments(T):
    """The split router with per-segment prefix lengths (Top-k inside [0, K)
    of each token's segment): at 65 836 rows after 128-row router tiles by
    the four-tokens-per-wavefront Top-k, at 4096 after split router tiles by
    the one-token-per-wavefront Top-k; indices bit-exact and weights against
    the oracle on the GPU's logits."""
    sh = I.QWEN3_VL_MOE
    rp = I.router_params(sh, seed=5)
    x = I.tokens(sh, T, seed=T + 1)
    wp = torch.empty((3 * sh.d * sh.E,), dtype=torch.bfloat16, device="cuda")
    abi.moe_pack_router(dev(rp["w_r"]), wp)
    so = np.array([0, 7, T // 3, T // 3, T - 129, T], np.int32)  # an empty segment, short ones
    Ks = np.array([8, 50, 128, 3, 85], np.int32)  # 3 < k: raised to k
    logits, idx, w = f32((T, sh.E)), i32((T, sh.k)), f32((T, sh.k))
    abi.moe_route_packed(dev(x, torch.bfloat16), wp, dev(rp["bias"]), sh.k, logits, idx, w,
                         seg_offsets=dev(so), K_dev=dev(Ks), ws=ws_for(T, sh.E, sh.k, sh.d, n_seg=5))
    a_gpu = host(logits).astype(np.float64)
    gi, gw = host(idx), host(w)
    for s_, (lo, hi) in enumerate(zip(so[:-1], so[1:])):
        if hi == lo:
            continue
        K = int(np.clip(Ks[s_], sh.k, sh.E))
        ref_idx, ref_w = oracle.prefix_route(a_gpu[lo:hi], K, sh.k)
        np.testing.assert_array_equal(gi[lo:hi], ref_idx)
        np.testing.assert_allclose(gw[lo:hi], ref_w, rtol=2e-5, atol=1e-6)


# ---------------------------------------------------------------------------
# moe_calibrate_prefix: masses bitwise, K and order exact (Eqs. 8, 9, 11, 12)
# ---------------------------------------------------------------------------
def oracle_calibrate(idx, w, E, k, segs, p):
    n_seg = len(segs) - 1
    mass = np.zeros((n_seg, E))
    K = np.zeros(n_seg, np.int64)
    cases = []
    for s in range(n_seg):
        lo, hi = segs[s], segs[s + 1]
        mass[s] = oracle.activated_mass(idx[lo:hi], w[lo:hi].astype(np.float64), E)
        K[s] = oracle.prefix_length(mass[s], p, k)
        if hi > lo:
            cases.append(oracle.routed_mass(idx[lo:hi], w[lo:hi].astype(np.float64), E))
    order = oracle.mean_mass_order(np.array(cases))[0] if cases else np.arange(E)
    return mass, K, order


@pytest.mark.parametrize("T,E,k,segs,p", [
    (128, 16, 2, None, 0.9),
    (512, 128, 8, None, 0.9),
    (4096, 128, 8, None, 0.9),
    (64, 128, 8, "per_token", 0.85),
    (300, 128, 8, [0, 0, 100, 100, 299, 300], 0.7),
    (512, 128, 8, None, 1.0),
    (512, 128, 8, None, 1e-9),
    (700, 1000, 8, [0, 350, 700], 0.9),
    (0, 16, 2, None, 0.9),
])
def test_calibrate_prefix_exact(T, E, k, segs, p):
    idx, w = I.synthetic_routing(T, E, k, seed=T + E)
    if segs is None:
        segs = [0, T]
        seg_dev = None
    else:
        if segs == "per_token":
            segs = list(range(T + 1))
        seg_dev = dev(np.array(segs, np.int32))
    n_seg = len(segs) - 1
    mass = torch.full((n_seg, E), float("nan"), dtype=torch.float64, device="cuda")
    K, order = i32((n_seg,)), i32((E,))
    idx_d = dev(idx) if T else torch.empty((0, k), dtype=torch.int32, device="cuda")
    w_d = dev(w) if T else torch.empty((0, k), dtype=torch.float32, device="cuda")
    abi.moe_calibrate_prefix(idx_d, w_d, E, p, mass, ws_for(T, E, k, 8), K_out=K, order=order,
                             seg_offsets=seg_dev)
    rm, rK, ro = oracle_calibrate(idx, w, E, k, segs, p)
    gm = host(mass)
    np.testing.assert_array_equal(gm.view(np.uint64), rm.view(np.uint64))  # bitwise
    np.testing.assert_array_equal(host(K), rK)
    np.testing.assert_array_equal(host(order), ro)


@pytest.mark.parametrize("T,E,k", [(300, 16, 2), (1500, 128, 8)])
def test_calibrate_skips_out_of_range_entries(T, E, k):
    """Routing entries with an expert outside [0, E) add nothing to the
    masses: the result is bitwise that of the same routing with those
    entries' weights set to zero (sorted path, and the chunked path above
    8192 entries)."""
    idx, w = I.synthetic_routing(T, E, k, seed=T + 5)
    rng = np.random.default_rng(T)
    bad = rng.choice(idx.size, size=idx.size // 53, replace=False)
    idx_bad = idx.reshape(-1).copy()
    idx_bad[bad] = rng.choice([-1, E, E + 100], size=bad.size)
    w_clean = w.reshape(-1).copy()
    w_clean[bad] = 0.0
    idx_bad, w_clean = idx_bad.reshape(T, k), w_clean.reshape(T, k)
    mass = torch.full((1, E), float("nan"), dtype=torch.float64, device="cuda")
    K, order = i32((1,)), i32((E,))
    abi.moe_calibrate_prefix(dev(idx_bad), dev(w), E, 0.9, mass, ws_for(T, E, k, 8), K_out=K, order=order)
    rm, rK, ro = oracle_calibrate(idx, w_clean, E, k, [0, T], 0.9)
    np.testing.assert_array_equal(host(mass).view(np.uint64), rm.view(np.uint64))
    np.testing.assert_array_equal(host(K), rK)
    np.testing.assert_array_equal(host(order), ro)


def test_combine_skips_out_of_range_rows():
    """Slots whose row index lies outside [0, T*k) contribute nothing: the
    output equals the oracle's combine with those slots' weights at zero."""
    T, k, d = 300, 8, 256
    A = T * k
    y = I.synthetic_rows(A, d, "bf16", seed=11)
    ros = I.synthetic_permutation(A, seed=12).astype(np.int32)
    _, w = I.synthetic_routing(T, 16, k, seed=13)
    rng = np.random.default_rng(14)
    bad = rng.choice(A, size=A // 41, replace=False)
    ros_bad = ros.copy()
    ros_bad[bad] = rng.choice([-1, A, A + 5000], size=bad.size)
    w_clean = w.reshape(-1).copy()
    w_clean[bad] = 0.0
    out = torch.empty((T, d), dtype=torch.bfloat16, device="cuda")
    abi.moe_combine(dev(y, torch.bfloat16), dev(ros_bad), dev(w), out)
    ref = oracle.combine(y, ros, w_clean.reshape(T, k))
    assert rel_inf(host(out), ref) <= TOL["bf16"]
    assert row_rel(host(out), ref) <= TOL["bf16"]


def test_calibrate_worked_example_golden():
    import json, os
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "prefix_worked_example.json")))
    idx = dev(np.array(g["topk_idx"], np.int32))
    w = dev(np.array(g["topk_w"], np.float32))
    for c in g["cases"]:
        mass = torch.empty((1, g["E"]), dtype=torch.float64, device="cuda")
        K = i32((1,))
        abi.moe_calibrate_prefix(idx, w, g["E"], c["p"], mass, ws_for(4, g["E"], 1, 8), K_out=K)
        np.testing.assert_array_equal(host(mass)[0], g["mass"])
        assert int(host(K)[0]) == c["K"], c["why"]
    rr = g["prefix_reroute_at_p_0.75"]
    ii, ww = i32((4, 1)), f32((4, 1))
    abi.moe_route(None, None, None, 1, dev(np.array(rr["logits"], np.float32)), ii, ww,
                  K_dev=dev(np.array([1], np.int32)))
    np.testing.assert_array_equal(host(ii), rr["idx"])
    np.testing.assert_array_equal(host(ww), rr["w"])


# ---------------------------------------------------------------------------
# moe_calibrate_route_prefix: one call, bitwise the two calls it replaces
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("T,E,k,p", [
    (512, 128, 8, 0.9),    # one launch (4096 entries)
    (64, 128, 8, 0.85),    # one launch, decode-sized
    (1, 16, 2, 0.5),       # a single token
    (1024, 128, 8, 1.0),   # one launch at the 8192-entry limit, p = 1
    (37, 300, 5, 0.7),     # E > 256: eight values per lane
    (200, 256, 8, 0.9),    # 128 < E <= 256: rows of 16 lanes, 16 values per lane
    (150, 200, 20, 0.8),   # k > 16: one wavefront per token
    (300, 512, 16, 0.95),  # E = 512, the largest one-launch pool
    (2000, 64, 8, 0.9),    # 16000 entries: the two-launch path
    (100, 600, 4, 0.9),    # E > 512: the two-launch path
])
def test_calibrate_route_prefix_matches_two_calls(T, E, k, p):
    logits = I.logits_with_ties(T, E, seed=T + E, levels=64)
    lg = dev(logits)
    idx_f, w_f = i32((T, k)), torch.empty((T, k), dtype=torch.float32, device="cuda")
    abi.moe_route(None, None, None, k, lg, idx_f, w_f)
    mass_a = torch.empty((1, E), dtype=torch.float64, device="cuda")
    K_a = i32((1,))
    idx_a, w_a = i32((T, k)), torch.empty((T, k), dtype=torch.float32, device="cuda")
    ws = torch.empty(abi.moe_workspace_size(T, E, k, 64, 64, 1), dtype=torch.uint8, device="cuda")
    abi.moe_calibrate_prefix(idx_f, w_f, E, p, mass_a, ws, K_out=K_a)
    abi.moe_route(None, None, None, k, lg, idx_a, w_a, K_dev=K_a)
    mass_b = torch.full((1, E), -1.0, dtype=torch.float64, device="cuda")
    K_b = i32((1,))
    idx_b, w_b = i32((T, k)), torch.empty((T, k), dtype=torch.float32, device="cuda")
    abi.moe_calibrate_route_prefix(lg, idx_f, w_f, p, mass_b, K_b, idx_b, w_b)
    torch.cuda.synchronize()
    assert torch.equal(K_a, K_b)
    assert torch.equal(mass_a.view(torch.int64), mass_b.view(torch.int64))
    assert torch.equal(idx_a, idx_b)
    assert torch.equal(w_a.view(torch.int32), w_b.view(torch.int32))
    # and against the oracle's K on the same routing (Eqs. 11, 12)
    s = oracle.activated_mass(host(idx_f), host(w_f).astype(np.float64), E)
    assert int(K_b.cpu()[0]) == int(oracle.prefix_length(s, p, k))


# ---------------------------------------------------------------------------
# moe_route_rcep: router, full-pool Top-k, masses, K, prefix re-route and
# grouping of one invocation in one call, bitwise the separate calls
# ---------------------------------------------------------------------------
# up to 8192 entries: the router and Top-k, then calibration, re-route and
# the grouping in one launch (the last workgroup to finish sorts; one
# workgroup at 1 row, four at 63 and 64, five at 65, 64 at 1024); beyond:
# the separate launches
@pytest.mark.parametrize("shape,T", [("qwen", 512), ("qwen", 64), ("qwen", 1), ("qwen", 63), ("qwen", 65),
                                     ("qwen", 1024), ("qwen", 1025), ("qwen", 4096), ("e96", 333), ("d64", 50),
                                     ("e256", 300), ("e256", 40), ("e256k20", 100), ("e256k20", 500),
                                     ("e256k20", 30), ("qwen", 0)])
def test_route_rcep_matches_separate_calls(shape, T):
    sh = {"qwen": I.QWEN3_VL_MOE, "e96": E96_BF16, "d64": D64_BF16, "e256": E256_BF16,
          "e256k20": E256_K20}[shape]
    E, k, p = sh.E, sh.k, 0.9
    rp = I.router_params(sh, seed=9)
    x = dev(I.tokens(sh, max(T, 1), seed=T + 2)[:T], torch.bfloat16)
    wp = torch.empty((3 * sh.d * E,), dtype=torch.bfloat16, device="cuda")
    abi.moe_pack_router(dev(rp["w_r"]), wp)
    bias = dev(rp["bias"]) if rp["bias"] is not None else None
    ws = ws_for(T, E, k, sh.d)
    A = T * k

    def outs():
        return dict(logits=f32((T, E)), idx_full=i32((T, k)), w_full=f32((T, k)),
                    mass=torch.full((1, E), -1.0, dtype=torch.float64, device="cuda"), K=i32((1,)),
                    idx=i32((T, k)), w=f32((T, k)), counts=i32((E,)), offsets=i32((E + 1,)),
                    src=i32((A,)), ros=i32((A,)))

    a = outs()
    if T:  # the router rejects an empty x without rows to route
        abi.moe_route_packed(x, wp, bias, k, a["logits"], a["idx_full"], a["w_full"], ws=ws)
    abi.moe_calibrate_route_prefix(a["logits"], a["idx_full"], a["w_full"], p, a["mass"], a["K"], a["idx"],
                                   a["w"])
    abi.moe_dispatch(a["idx"], E, None, a["counts"], a["offsets"], a["src"], a["ros"], None, ws)
    b = outs()
    abi.moe_route_rcep(x, wp, bias, k, p, b["logits"], b["idx_full"], b["w_full"], b["mass"], b["K"], b["idx"],
                       b["w"], b["counts"], b["offsets"], b["src"], b["ros"], ws)
    torch.cuda.synchronize()
    for n in a:
        assert torch.equal(a[n].view(torch.uint8), b[n].view(torch.uint8)), n
    K = int(host(b["K"])[0])
    if T == 0:
        assert K == k and (host(b["counts"]) == 0).all() and (host(b["offsets"]) == 0).all()
        return
    # and against the oracle on the same logits (Eqs. 11, 12, Algorithm 1)
    lg = host(b["logits"]).astype(np.float64)
    s = oracle.activated_mass(host(b["idx_full"]), host(b["w_full"]).astype(np.float64), E)
    assert K == int(oracle.prefix_length(s, p, k))
    ref_idx, ref_w = oracle.prefix_route(lg, K, k)
    np.testing.assert_array_equal(host(b["idx"]), ref_idx)
    np.testing.assert_allclose(host(b["w"]), ref_w, rtol=2e-5, atol=1e-6)
    rc, ro, rs, rr = oracle.dispatch(ref_idx, E)
    np.testing.assert_array_equal(host(b["counts"]), rc)
    np.testing.assert_array_equal(host(b["offsets"]), ro)
    np.testing.assert_array_equal(host(b["src"]), rs)
    np.testing.assert_array_equal(host(b["ros"]), rr)


# ---------------------------------------------------------------------------
# moe_rcep_layer: one RCEP layer (routing, expert FFN over the prefix,
# combine and residual) in one call, bitwise the three calls it stands for
# ---------------------------------------------------------------------------
D256_E64 = I.LayerShape(d=256, E=64, m=256, k=4, dtype="bf16", zipf_alpha=0.35)
D256_E256_K20 = I.LayerShape(d=256, E=256, m=256, k=20, dtype="bf16", zipf_alpha=0.35)
RCEP_LAYER_SHAPES = {"qwen": I.QWEN3_VL_MOE, "e64": D256_E64, "e256k20": D256_E256_K20}


class _RcepLayer:
    """Weights of one shape and the outputs of one call."""

    def __init__(self, sh, seed):
        self.sh = sh
        rp = I.router_params(sh, seed=seed)
        prm = I.layer_params(sh, seed=seed + 1)
        self.rp, self.prm = rp, prm
        self.wp = torch.empty((3 * sh.d * sh.E,), dtype=torch.bfloat16, device="cuda")
        abi.moe_pack_router(dev(rp["w_r"]), self.wp)
        self.bias = dev(rp["bias"]) if rp["bias"] is not None else None
        wgu, wd = dev(prm["w_gate_up"], torch.bfloat16), dev(prm["w_down"], torch.bfloat16)
        self.wgu_p, self.wd_p = torch.empty_like(wgu), torch.empty_like(wd)
        abi.moe_pack_expert_weights(wgu, self.wgu_p)
        abi.moe_pack_expert_weights(wd, self.wd_p)

    def outs(self, T):
        E, k, d = self.sh.E, self.sh.k, self.sh.d
        A = T * k
        return dict(logits=f32((T, E)), idx_full=i32((T, k)), w_full=f32((T, k)),
                    mass=torch.full((1, E), -1.0, dtype=torch.float64, device="cuda"), K=i32((1,)),
                    idx=i32((T, k)), w=f32((T, k)), counts=i32((E,)), offsets=i32((E + 1,)),
                    src=i32((A,)), ros=i32((A,)),
                    y=torch.full((A, d), 7.0, dtype=torch.bfloat16, device="cuda"))

    def separate(self, x, residual, p, ws):
        o = self.outs(x.shape[0])
        abi.moe_route_rcep(x, self.wp, self.bias, self.sh.k, p, o["logits"], o["idx_full"], o["w_full"], o["mass"],
                           o["K"], o["idx"], o["w"], o["counts"], o["offsets"], o["src"], o["ros"], ws)
        o["out"] = torch.full_like(x, 5.0)
        if x.shape[0]:
            abi.moe_expert_ffn_packed_gather(x, self.sh.k, o["src"], o["offsets"], self.wgu_p, self.wd_p, o["y"],
                                             ws, K_dev=o["K"])
            if residual is None:
                abi.moe_combine(o["y"], o["ros"], o["w"], o["out"])
            else:
                abi.moe_combine_residual(o["y"], o["ros"], o["w"], residual, o["out"])
        return o

    def routed(self, x, p, ws, o=None):
        """The routing and expert FFN of one call, no combine."""
        o = o if o is not None else self.outs(x.shape[0])
        abi.moe_route_rcep(x, self.wp, self.bias, self.sh.k, p, o["logits"], o["idx_full"], o["w_full"], o["mass"],
                           o["K"], o["idx"], o["w"], o["counts"], o["offsets"], o["src"], o["ros"], ws)
        abi.moe_expert_ffn_packed_gather(x, self.sh.k, o["src"], o["offsets"], self.wgu_p, self.wd_p, o["y"], ws,
                                         K_dev=o["K"])
        return o

    def chained(self, prev, h, p, ws, o=None):
        o = o if o is not None else self.outs(h.shape[0])
        pv = (prev["y"], prev["ros"], prev["w"]) if prev is not None else None
        abi.moe_rcep_layer_chained(pv, h, self.wp, self.bias, self.sh.k, p, self.wgu_p, self.wd_p, o["logits"],
                                   o["idx_full"], o["w_full"], o["mass"], o["K"], o["idx"], o["w"], o["counts"],
                                   o["offsets"], o["src"], o["ros"], o["y"], ws)
        return o

    def layer(self, x, residual, out, p, ws, guard=None):
        o = self.outs(x.shape[0])
        abi.moe_rcep_layer(x, self.wp, self.bias, self.sh.k, p, self.wgu_p, self.wd_p, residual, out,
                           o["logits"], o["idx_full"], o["w_full"], o["mass"], o["K"], o["idx"], o["w"],
                           o["counts"], o["offsets"], o["src"], o["ros"], o["y"], ws, guard=guard)
        o["out"] = out
        return o


def _assert_same(a, b, names):
    for n in names:
        assert torch.equal(a[n].contiguous().view(torch.uint8), b[n].contiguous().view(torch.uint8)), n


ALL_OUTS = ("logits", "idx_full", "w_full", "mass", "K", "idx", "w", "counts", "offsets", "src", "ros", "y",
            "out")


# T*k <= 8192: the routing's one-launch grouping also clears the expert
# FFN's counters (qwen 1, 64, 512, 1024; e64; e256k20); beyond, the
# separate launches with the FFN's own clearing (qwen 1025, e64 2100)
# (no_res: residual NULL, the plain combine)
@pytest.mark.parametrize("shape,T,no_res", [("qwen", 512, False), ("qwen", 64, False), ("qwen", 1, False),
                                            ("qwen", 1024, False), ("qwen", 1025, False), ("e64", 300, False),
                                            ("e64", 2100, False), ("e256k20", 100, False), ("e64", 0, False),
                                            ("qwen", 512, True), ("qwen", 1025, True), ("e64", 300, True)])
def test_rcep_layer_matches_separate_calls(shape, T, no_res):
    sh = RCEP_LAYER_SHAPES[shape]
    L = _RcepLayer(sh, seed=13)
    p = 0.9
    x = dev(I.tokens(sh, max(T, 1), seed=T + 5)[:T], torch.bfloat16)
    residual = None if no_res else dev(I.synthetic_rows(max(T, 1), sh.d, "bf16", seed=T + 6)[:T], torch.bfloat16)
    ws = ws_for(T, sh.E, sh.k, sh.d, sh.m)
    a = L.separate(x, residual, p, ws)
    ws.fill_(0xA5)  # the composed call starts from a workspace holding stale counters
    b = L.layer(x, residual, torch.full_like(x, 5.0), p, ws)
    torch.cuda.synchronize()
    if T == 0:
        assert int(host(b["K"])[0]) == sh.k and (host(b["counts"]) == 0).all()
        _assert_same(a, b, ("mass", "K", "counts", "offsets"))
        return
    assert_ffn_ran_all(ws)
    _assert_same(a, b, ALL_OUTS)
    K = int(host(b["K"])[0])
    assert K == int(oracle.prefix_length(
        oracle.activated_mass(host(b["idx_full"]), host(b["w_full"]).astype(np.float64), sh.E), p, sh.k))
    if shape != "qwen" or T <= 64:
        # against the oracle's layer on the same logits and K (Algorithm 2,
        # Eqs. 10-12 and App. A.3 Eq. 15), plus the residual
        ref = oracle.moe_layer_rcep(host(x), L.rp["w_r"], L.rp["bias"], L.prm["w_gate_up"], L.prm["w_down"],
                                    sh.k, p, logits=host(b["logits"]), K_override=[K])
        np.testing.assert_array_equal(host(b["idx"]), ref["idx"])
        want = ref["out"] if residual is None else host(residual).astype(np.float64) + ref["out"]
        assert rel_inf(host(b["out"]), want) <= TOL["bf16"]
        assert row_rel(host(b["out"]), want) <= TOL["bf16"]


def _dense_outs(T, sh):
    E, k, d = sh.E, sh.k, sh.d
    A = T * k
    return dict(logits=f32((T, E)), idx=i32((T, k)), w=f32((T, k)), counts=i32((E,)), offsets=i32((E + 1,)),
                src=i32((A,)), ros=i32((A,)), y=torch.full((A, d), 7.0, dtype=torch.bfloat16, device="cuda"))


DENSE_OUTS = ("logits", "idx", "w", "counts", "offsets", "src", "ros", "y", "out")


# T*k <= 8192: the one-workgroup grouping (qwen 1, 64, 1024; e64; e256k20);
# up to 64 chunks of 1024 entries the fused scan and rank (qwen 1025, 4096),
# beyond, histogram, scan and rank launches (qwen 9000)
@pytest.mark.parametrize("shape,T,no_res", [("qwen", 64, False), ("qwen", 1, False), ("qwen", 1024, False),
                                            ("qwen", 1025, False), ("qwen", 4096, True), ("qwen", 9000, False),
                                            ("e64", 300, True), ("e256k20", 100, False), ("e64", 0, False)])
def test_dense_layer_matches_separate_calls(shape, T, no_res):
    """moe_dense_layer against moe_route_packed + moe_dispatch + the
    gathering expert FFN + the combine (with the residual, or without):
    bitwise every output, on a workspace left holding stale counters, and
    the FFN ran every item with no clearing launch of its own."""
    sh = RCEP_LAYER_SHAPES[shape]
    L = _RcepLayer(sh, seed=31)
    x = dev(I.tokens(sh, max(T, 1), seed=T + 11)[:T], torch.bfloat16)
    residual = None if no_res else dev(I.synthetic_rows(max(T, 1), sh.d, "bf16", seed=T + 12)[:T], torch.bfloat16)
    ws = ws_for(T, sh.E, sh.k, sh.d, sh.m)
    a = _dense_outs(T, sh)
    a["out"] = torch.full_like(x, 5.0)
    if T:
        abi.moe_route_packed(x, L.wp, L.bias, sh.k, a["logits"], a["idx"], a["w"], ws=ws)
    abi.moe_dispatch(a["idx"], sh.E, None, a["counts"], a["offsets"], a["src"], a["ros"], None, ws)
    if T:
        abi.moe_expert_ffn_packed_gather(x, sh.k, a["src"], a["offsets"], L.wgu_p, L.wd_p, a["y"], ws)
        if residual is None:
            abi.moe_combine(a["y"], a["ros"], a["w"], a["out"])
        else:
            abi.moe_combine_residual(a["y"], a["ros"], a["w"], residual, a["out"])
    torch.cuda.synchronize()
    ws.fill_(0xA5)
    b = _dense_outs(T, sh)
    b["out"] = torch.full_like(x, 5.0)
    abi.moe_dense_layer(x, L.wp, L.bias, sh.k, L.wgu_p, L.wd_p, residual, b["out"], b["logits"], b["idx"], b["w"],
                        b["counts"], b["offsets"], b["src"], b["ros"], b["y"], ws)
    torch.cuda.synchronize()
    if T == 0:
        _assert_same(a, b, ("counts", "offsets"))
        return
    path, _ = assert_ffn_ran_all(ws)
    assert path == abi.FFN_PATH_PERSISTENT
    _assert_same(a, b, DENSE_OUTS)


# qwen 1, 64, 512, e64: the previous combine inside the router's launch;
# qwen 1025 (T*k > 8192) and e256k20 (E > 128): the combine on its own first
@pytest.mark.parametrize("shape,T", [("qwen", 64), ("qwen", 512), ("qwen", 1), ("qwen", 1025), ("e64", 300),
                                     ("e256k20", 100)])
@pytest.mark.parametrize("shared", [False, True])
def test_rcep_layer_chained_matches_separate_calls(shape, T, shared):
    """Two layers through moe_rcep_layer_chained (the first without a
    previous layer, the second combining the first's expert outputs into h
    before its routing) against moe_route_rcep + the expert FFN and
    moe_combine_residual between them: bitwise every output and h.  With
    `shared` the second call writes the arrays the first wrote (a stack's
    one set of buffers), on a workspace left holding stale counters."""
    sh = RCEP_LAYER_SHAPES[shape]
    L0, L1 = _RcepLayer(sh, seed=23), _RcepLayer(sh, seed=29)
    p = 0.9
    x = dev(I.tokens(sh, T, seed=T + 9), torch.bfloat16)
    ws = ws_for(T, sh.E, sh.k, sh.d, sh.m)
    h_ref = x.clone()
    a0 = L0.routed(h_ref, p, ws)
    abi.moe_combine_residual(a0["y"], a0["ros"], a0["w"], h_ref, h_ref)
    a1 = L1.routed(h_ref, p, ws)
    torch.cuda.synchronize()
    a0 = {n: v.clone() for n, v in a0.items()}
    ws.fill_(0xA5)
    h = x.clone()
    b0 = L0.chained(None, h, p, ws)
    torch.cuda.synchronize()
    assert_ffn_ran_all(ws)
    _assert_same(a0, b0, ALL_OUTS[:-1])
    assert torch.equal(h.view(torch.uint8), x.view(torch.uint8))
    b1 = L1.chained(b0, h, p, ws, o=b0 if shared else None)
    torch.cuda.synchronize()
    assert_ffn_ran_all(ws)
    assert torch.equal(h.view(torch.uint8), h_ref.view(torch.uint8))
    _assert_same(a1, b1, ALL_OUTS[:-1])


@pytest.mark.parametrize("shape,T", [("qwen", 64), ("qwen", 1025), ("e64", 300)])
def test_rcep_layer_in_place_and_reused_workspace(shape, T):
    """out == residual == x (the hidden state updated in place), on one
    workspace reused by a larger then a smaller call: bitwise the separate
    calls each time, and the expert FFN ran every item."""
    sh = RCEP_LAYER_SHAPES[shape]
    L = _RcepLayer(sh, seed=17)
    ws = ws_for(2 * T, sh.E, sh.k, sh.d, sh.m)
    for n in (2 * T, T):
        h = dev(I.tokens(sh, n, seed=n + 3), torch.bfloat16)
        a = L.separate(h, h, 0.9, ws)
        b = L.layer(h, h, h, 0.9, ws)
        torch.cuda.synchronize()
        assert_ffn_ran_all(ws)
        _assert_same(a, b, ALL_OUTS)


def test_rcep_layer_guard():
    """moe_rcep_layer_if: with the value inside the range the results of
    the plain call; outside it nothing is written, moe_ffn_status still
    reports the previous call."""
    sh = D256_E64
    T = 300
    L = _RcepLayer(sh, seed=19)
    x = dev(I.tokens(sh, T, seed=1), torch.bfloat16)
    res = dev(I.synthetic_rows(T, sh.d, "bf16", seed=2), torch.bfloat16)
    ws = ws_for(T, sh.E, sh.k, sh.d, sh.m)
    g = dev(np.array([3], np.int32))
    a = L.layer(x, res, torch.full_like(x, 5.0), 0.9, ws)
    b = L.layer(x, res, torch.full_like(x, 5.0), 0.9, ws, guard=(g, 3, 4))
    torch.cuda.synchronize()
    _assert_same(a, b, ALL_OUTS)
    st0 = torch.full((4,), -1, dtype=torch.int32, device="cuda")
    abi.moe_ffn_status(ws, st0)
    c = L.layer(x, res, torch.full_like(x, 5.0), 0.9, ws, guard=(g, 4, 8))
    st1 = torch.full((4,), -1, dtype=torch.int32, device="cuda")
    abi.moe_ffn_status(ws, st1)
    torch.cuda.synchronize()
    assert (host(c["out"]).astype(np.float32) == 5.0).all()
    assert (host(c["K"]) == -7).all() and (host(c["counts"]) == -7).all()
    assert (host(c["mass"]) == -1.0).all()
    assert torch.equal(st0, st1)


# ---------------------------------------------------------------------------
# moe_dispatch: bit-exact counting sort and bitwise gather
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("T,E,k,d,dt,K", [
    (512, 16, 2, 256, "f32", None),
    (4096, 128, 8, 2048, "bf16", None),
    (512, 128, 8, 2048, "bf16", 84),
    (1, 128, 8, 2048, "bf16", None),
    (37, 7, 3, 24, "f32", None),
    (3000, 1000, 4, 64, "bf16", None),
    (129, 5, 5, 6, "bf16", None),
    (1000, 64, 2, 10, "f32", None),
    # more than 8192 assignments (also 4096 x 8 and 3000 x 4 above): the
    # multi-workgroup path, histograms then ranks with the scan folded in
    # (up to 64 chunks of 1024: 8192 x 8 is the largest), or histograms,
    # scan and ranks as three launches beyond that
    (8192, 128, 8, 64, "bf16", None),
    (9000, 128, 8, 64, "bf16", None),
    (8193, 1000, 8, 16, "f32", 999),
])
def test_dispatch_exact(T, E, k, d, dt, K):
    idx, _ = I.synthetic_routing(T, E, k, seed=3 * T + E, K=K)
    x = I.synthetic_rows(T, d, dt, seed=T + d)
    A = T * k
    counts, offsets = i32((E,)), i32((E + 1,))
    src, ros = i32((A,)), i32((A,))
    xp = torch.zeros((A, d), dtype=TDT[dt], device="cuda")
    ws = torch.empty(abi.moe_workspace_size(T, E, k, d, 64, 1), dtype=torch.uint8, device="cuda")
    abi.moe_dispatch(dev(idx), E, dev(x, TDT[dt]), counts, offsets, src, ros, xp, ws)
    rc, ro, rs, rr = oracle.dispatch(idx, E)
    np.testing.assert_array_equal(host(counts), rc)
    np.testing.assert_array_equal(host(offsets), ro)
    np.testing.assert_array_equal(host(src), rs)
    np.testing.assert_array_equal(host(ros), rr)
    if K is not None:
        assert (host(counts)[K:] == 0).all()
    ref_xp = x[rs // k]
    np.testing.assert_array_equal(host(xp).view(np.uint32), ref_xp.view(np.uint32))


@pytest.mark.parametrize("T", [1000, 4096, 9000])
def test_dispatch_drops_out_of_range_entries(T):
    """Entries outside [0, E) get no row and row_of_slot -1; the valid ones
    are grouped as a stable sort of the valid entries alone (one workgroup,
    histograms then ranks with the scan folded in, and three launches)."""
    E, k, d = 128, 8, 64
    idx, _ = I.synthetic_routing(T, E, k, seed=T)
    flat = idx.reshape(-1).copy()
    rng = np.random.default_rng(T)
    bad = rng.choice(flat.size, size=flat.size // 97, replace=False)
    flat[bad] = rng.choice([-1, E, 1000, -7], size=bad.size)
    idx = flat.reshape(T, k)
    x = I.synthetic_rows(T, d, "bf16", seed=T + 1)
    A = T * k
    counts, offsets = i32((E,)), i32((E + 1,))
    src, ros = i32((A,)), i32((A,))
    xp = torch.zeros((A, d), dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(abi.moe_workspace_size(T, E, k, d, 64, 1), dtype=torch.uint8, device="cuda")
    abi.moe_dispatch(dev(idx), E, dev(x, torch.bfloat16), counts, offsets, src, ros, xp, ws)
    valid = (flat >= 0) & (flat < E)
    a_valid = np.nonzero(valid)[0]
    order = a_valid[np.argsort(flat[a_valid], kind="stable")]
    n = order.size
    np.testing.assert_array_equal(host(counts), np.bincount(flat[a_valid], minlength=E))
    np.testing.assert_array_equal(host(offsets), np.concatenate([[0], np.cumsum(host(counts))]))
    assert int(host(offsets)[E]) == n < A
    np.testing.assert_array_equal(host(src)[:n], order)
    ro = host(ros)
    assert (ro[~valid] == -1).all()
    np.testing.assert_array_equal(ro[order], np.arange(n))
    np.testing.assert_array_equal(host(xp)[:n].view(np.uint32), x[order // k].view(np.uint32))


def test_dispatch_empty():
    counts, offsets = i32((16,)), i32((17,))
    e = torch.empty((0,), dtype=torch.int32, device="cuda")
    ws = torch.empty(256, dtype=torch.uint8, device="cuda")
    abi.moe_dispatch(torch.empty((0, 2), dtype=torch.int32, device="cuda"), 16, None, counts,
                     offsets, e, e, None, ws)
    assert (host(counts) == 0).all() and (host(offsets) == 0).all()


# ---------------------------------------------------------------------------
# moe_expert_ffn: SwiGLU per dispatched row
# ---------------------------------------------------------------------------
FFN_CASES = [
    # E, d, m, dtype, rows, K (experts evaluated), special counts
    (16, 256, 128, "f32", 1024, None, None),
    (8, 2048, 768, "bf16", 1500, None, [0, 1, 127, 128, 129, 300, 700, 115]),
    (6, 2048, 768, "bf16", 900, 4, None),
    (3, 256, 128, "bf16", 300, None, [255, 0, 45]),
    (128, 256, 128, "bf16", 4096, None, None),
    (5, 40, 12, "f32", 77, None, None),
]


@pytest.mark.parametrize("E,d,m,dt,rows,K,cnt", FFN_CASES)
def test_expert_ffn(E, d, m, dt, rows, K, cnt):
    sh = I.LayerShape(d=d, E=E, m=m, k=1, dtype=dt)
    prm = I.layer_params(sh, seed=E + d)
    counts = np.array(cnt, np.int64) if cnt is not None else I.synthetic_counts(E, rows, seed=rows)
    rows = int(counts.sum())
    offsets = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    xp = I.synthetic_rows(rows, d, dt, seed=rows + 1)
    expert_of_row = np.repeat(np.arange(E), counts)
    y = torch.full((rows, d), 7.0, dtype=TDT[dt], device="cuda")
    ws = torch.empty(abi.moe_workspace_size(rows, E, 1, d, m, 1), dtype=torch.uint8, device="cuda")
    K_dev = dev(np.array([K], np.int32)) if K is not None else None
    abi.moe_expert_ffn(dev(xp, TDT[dt]), dev(offsets), dev(prm["w_gate_up"], TDT[dt]),
                       dev(prm["w_down"], TDT[dt]), y, ws, K_dev=K_dev)
    path, _ = assert_ffn_ran_all(ws)
    assert path == (abi.FFN_PATH_F32 if dt == "f32" else abi.FFN_PATH_ROW_MAJOR)
    got = host(y)
    live = expert_of_row < (K if K is not None else E)
    ref = oracle.expert_ffn_rows(xp[live], expert_of_row[live], prm["w_gate_up"], prm["w_down"])
    assert rel_inf(got[live], ref) <= TOL[dt]
    assert row_rel(got[live], ref) <= TOL[dt]
    assert (got[~live] == 7.0).all()  # experts >= K are not evaluated


# ---------------------------------------------------------------------------
# packed expert weights: layout, then the packed FFN against the row-major one
# ---------------------------------------------------------------------------
def packed_layout(w):
    """The documented fragment layout, written with reshapes: element (e, r, c)
    goes to e*R*C + ((c//16)*(R//32) + r//32)*512 + 8*(r%32 + 32*((c%16)//8)) + c%8."""
    E, R, C = w.shape
    v = w.reshape(E, R // 32, 32, C // 16, 2, 8)          # e, rb, r, kb, h, c
    return np.ascontiguousarray(v.transpose(0, 3, 1, 4, 2, 5)).reshape(E, R, C)  # e, kb, rb, h, r, c


@pytest.mark.parametrize("E,R,C", [(3, 64, 48), (2, 1536, 2048), (5, 2048, 768), (1, 32, 16)])
def test_pack_expert_weights_layout(E, R, C):
    rng = np.random.default_rng(R + C)
    w = rng.integers(0, 1 << 16, size=(E, R, C), dtype=np.uint16)
    wt = dev(w.view(np.int16)).view(torch.bfloat16)
    out = torch.empty_like(wt)
    abi.moe_pack_expert_weights(wt, out)
    torch.cuda.synchronize()
    got = out.view(torch.int16).cpu().numpy().view(np.uint16)
    assert np.array_equal(got, packed_layout(w))


# token-tile distributions for the persistent kernel's per-XCD split: one
# expert holding every row (128-row tiles), a single tile, more XCDs than
# tiles, empty experts between full ones, and a prefix K with no rows past it
SKEW_CASES = [
    (128, 2048, 768, "bf16", 4096, None, [0] * 5 + [4096] + [0] * 122),  # 64-row tiles (< 48 rows per expert)
    (8, 2048, 768, "bf16", 4096, None, [0, 0, 0, 4096, 0, 0, 0, 0]),       # 128-row tiles
    (8, 512, 256, "bf16", 20, None, [0, 0, 0, 20, 0, 0, 0, 0]),
    (4, 512, 256, "bf16", 130, None, [0, 65, 0, 65]),
    (32, 512, 256, "bf16", 6000, None, [1500, 0, 0, 1500, 0, 1500] + [0] * 25 + [1500]),
    (16, 512, 256, "bf16", 3000, 5, [600, 600, 600, 600, 600] + [0] * 11),
    (1000, 256, 256, "bf16", 700, None, None),                        # 1000 experts, mostly empty
]

PACKED_CASES = [c for c in FFN_CASES if c[3] == "bf16" and c[2] % 256 == 0] + SKEW_CASES + [
    (4, 512, 256, "bf16", 700, None, [300, 0, 1, 399]),  # one 8-k-step body, ragged tails
    (2, 2048, 768, "bf16", 1700, None, [1600, 100]),       # many tiles of one expert
    # few rows per expert (decode-like weight streaming)
    (128, 2048, 768, "bf16", 512, None, None),             # 64 tokens x top-8
    (16, 512, 256, "bf16", 200, None, [0, 1, 31, 32, 33, 63, 40] + [0] * 9),  # ragged tails
    (6, 2048, 768, "bf16", 60, 4, None),                   # experts >= K skipped
]


@pytest.mark.parametrize("E,d,m,dt,rows,K,cnt", PACKED_CASES)
def test_expert_ffn_packed(E, d, m, dt, rows, K, cnt):
    sh = I.LayerShape(d=d, E=E, m=m, k=1, dtype=dt)
    prm = I.layer_params(sh, seed=E + d)
    counts = np.array(cnt, np.int64) if cnt is not None else I.synthetic_counts(E, rows, seed=rows)
    rows = int(counts.sum())
    offsets = dev(np.concatenate([[0], np.cumsum(counts)]).astype(np.int32))
    xp = dev(I.synthetic_rows(rows, d, dt, seed=rows + 1), TDT[dt])
    wgu, wd = dev(prm["w_gate_up"], TDT[dt]), dev(prm["w_down"], TDT[dt])
    wgu_p, wd_p = torch.empty_like(wgu), torch.empty_like(wd)
    abi.moe_pack_expert_weights(wgu, wgu_p)
    abi.moe_pack_expert_weights(wd, wd_p)
    ws = torch.empty(abi.moe_workspace_size(rows, E, 1, d, m, 1), dtype=torch.uint8, device="cuda")
    K_dev = dev(np.array([K], np.int32)) if K is not None else None
    y_ref = torch.full((rows, d), 7.0, dtype=TDT[dt], device="cuda")
    y = torch.full((rows, d), 7.0, dtype=TDT[dt], device="cuda")
    abi.moe_expert_ffn(xp, offsets, wgu, wd, y_ref, ws, K_dev=K_dev)
    abi.moe_expert_ffn_packed(xp, offsets, wgu_p, wd_p, y, ws, K_dev=K_dev)
    path, planned = assert_ffn_ran_all(ws)
    assert path == abi.FFN_PATH_PERSISTENT and (planned > 0) == (rows > 0)
    # same fragments, same k order, same float32 accumulation: bitwise equal
    assert torch.equal(y.view(torch.int16), y_ref.view(torch.int16))
    expert_of_row = np.repeat(np.arange(E), counts)
    live = expert_of_row < (K if K is not None else E)
    ref = oracle.expert_ffn_rows(host(xp)[live], expert_of_row[live], prm["w_gate_up"], prm["w_down"])
    assert rel_inf(host(y)[live], ref) <= TOL[dt]
    assert row_rel(host(y)[live], ref) <= TOL[dt]
    assert (host(y)[~live] == 7.0).all()  # experts >= K are not evaluated


def test_expert_ffn_clamps_offsets_to_rows_max():
    """Offsets past rows_max are clamped: expert e evaluates rows
    [min(off[e], R), min(off[e + 1], R)), so the experts beyond R get no rows
    (row-major and packed paths, bitwise equal, and against the oracle)."""
    E, d, m, R = 8, 256, 256, 300
    sh = I.LayerShape(d=d, E=E, m=m, k=1, dtype="bf16")
    prm = I.layer_params(sh, seed=77)
    raw = np.array([0, 50, 120, 120, 200, 260, 400, 500, 600], np.int32)
    xp = dev(I.synthetic_rows(R, d, "bf16", seed=78), torch.bfloat16)
    wgu, wd = dev(prm["w_gate_up"], torch.bfloat16), dev(prm["w_down"], torch.bfloat16)
    wgu_p, wd_p = torch.empty_like(wgu), torch.empty_like(wd)
    abi.moe_pack_expert_weights(wgu, wgu_p)
    abi.moe_pack_expert_weights(wd, wd_p)
    ws = torch.empty(abi.moe_workspace_size(R, E, 1, d, m, 1), dtype=torch.uint8, device="cuda")
    y_ref = torch.full((R, d), 7.0, dtype=torch.bfloat16, device="cuda")
    y = torch.full((R, d), 7.0, dtype=torch.bfloat16, device="cuda")
    abi.moe_expert_ffn(xp, dev(raw), wgu, wd, y_ref, ws)
    abi.moe_expert_ffn_packed(xp, dev(raw), wgu_p, wd_p, y, ws)
    assert torch.equal(y.view(torch.int16), y_ref.view(torch.int16))
    off = np.minimum(raw, R)
    expert_of_row = np.repeat(np.arange(E), np.diff(off))
    assert expert_of_row.size == R
    ref = oracle.expert_ffn_rows(host(xp), expert_of_row, prm["w_gate_up"], prm["w_down"])
    assert rel_inf(host(y), ref) <= TOL["bf16"]


# ---------------------------------------------------------------------------
# moe_expert_ffn_packed_gather: the dispatch gather inside the GEMM
# ---------------------------------------------------------------------------
GATHER_CASES = [
    # T, E, k, d, m, K
    (512, 128, 8, 2048, 768, None),   # 512 text rows, full pool (64-row tiles: < 48 rows per expert)
    (512, 128, 8, 2048, 768, 84),     # prefix of 84 experts
    (1024, 128, 8, 2048, 768, None),  # 1024 rows (128-row tiles, 64 rows per expert)
    (4096, 128, 8, 2048, 768, None),  # 4096 rows (128-row tiles)
    (37, 6, 3, 512, 256, None),       # ragged, few experts
    (1, 16, 2, 256, 256, None),       # a single token
    (300, 4, 2, 512, 256, 3),         # experts >= K skipped
]


@pytest.mark.parametrize("T,E,k,d,m,K", GATHER_CASES)
def test_expert_ffn_packed_gather(T, E, k, d, m, K):
    sh = I.LayerShape(d=d, E=E, m=m, k=k, dtype="bf16")
    prm = I.layer_params(sh, seed=E + d + k)
    idx, _ = I.synthetic_routing(T, E, k, seed=T + 11 * E, K=K)
    assert idx.shape == (T, k)
    x = dev(I.synthetic_rows(T, d, "bf16", seed=T + d), torch.bfloat16)
    A = T * k
    counts, offsets, src, ros = i32((E,)), i32((E + 1,)), i32((A,)), i32((A,))
    xp = torch.empty((A, d), dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(abi.moe_workspace_size(T, E, k, d, m, 1), dtype=torch.uint8, device="cuda")
    wgu, wd = dev(prm["w_gate_up"], torch.bfloat16), dev(prm["w_down"], torch.bfloat16)
    wgu_p, wd_p = torch.empty_like(wgu), torch.empty_like(wd)
    abi.moe_pack_expert_weights(wgu, wgu_p)
    abi.moe_pack_expert_weights(wd, wd_p)
    K_dev = dev(np.array([K], np.int32)) if K is not None else None
    y_ref = torch.full((A, d), 7.0, dtype=torch.bfloat16, device="cuda")
    y = torch.full((A, d), 7.0, dtype=torch.bfloat16, device="cuda")
    abi.moe_dispatch(dev(idx), E, x, counts, offsets, src, ros, xp, ws)
    abi.moe_expert_ffn_packed(xp, offsets, wgu_p, wd_p, y_ref, ws, K_dev=K_dev)
    # the same dispatch without the row copy, then the gathering GEMM
    counts2, offsets2, src2, ros2 = i32((E,)), i32((E + 1,)), i32((A,)), i32((A,))
    abi.moe_dispatch(dev(idx), E, None, counts2, offsets2, src2, ros2, None, ws)
    assert torch.equal(src2, src) and torch.equal(offsets2, offsets)
    abi.moe_expert_ffn_packed_gather(x, k, src2, offsets2, wgu_p, wd_p, y, ws, K_dev=K_dev)
    assert_ffn_ran_all(ws)
    assert torch.equal(y.view(torch.int16), y_ref.view(torch.int16))
    # against the oracle on every live row
    rs = host(src)
    e_of_row = np.repeat(np.arange(E), host(counts))
    live = np.flatnonzero(e_of_row < (K if K is not None else E))
    ref = oracle.expert_ffn_rows(host(x)[rs[live] // k], e_of_row[live], prm["w_gate_up"], prm["w_down"])
    assert rel_inf(host(y)[live], ref) <= TOL["bf16"]
    assert row_rel(host(y)[live], ref) <= TOL["bf16"]


@pytest.mark.parametrize("shift", [16, 48, 112])
def test_expert_ffn_packed_gather_unaligned_workspace(shift):
    """A workspace that starts 16 bytes (not 256) into an allocation gives
    the bits of an aligned one: the library rounds its h and counters up to
    a 256-byte boundary, so no h line is shared between token tiles."""
    T, E, k, d, m = 1024, 32, 4, 512, 256
    sh = I.LayerShape(d=d, E=E, m=m, k=k, dtype="bf16")
    prm = I.layer_params(sh, seed=31)
    idx, _ = I.synthetic_routing(T, E, k, seed=32)
    x = dev(I.synthetic_rows(T, d, "bf16", seed=33), torch.bfloat16)
    A = T * k
    counts, offsets, src, ros = i32((E,)), i32((E + 1,)), i32((A,)), i32((A,))
    nb = abi.moe_workspace_size(T, E, k, d, m, 1)
    ws = torch.empty(nb, dtype=torch.uint8, device="cuda")
    big = torch.empty(nb + 256, dtype=torch.uint8, device="cuda")
    ws_shift = big[shift:shift + nb]
    assert ws_shift.data_ptr() % 256 == shift
    abi.moe_dispatch(dev(idx), E, None, counts, offsets, src, ros, None, ws)
    wgu, wd = dev(prm["w_gate_up"], torch.bfloat16), dev(prm["w_down"], torch.bfloat16)
    wgu_p, wd_p = torch.empty_like(wgu), torch.empty_like(wd)
    abi.moe_pack_expert_weights(wgu, wgu_p)
    abi.moe_pack_expert_weights(wd, wd_p)
    y1 = torch.full((A, d), 7.0, dtype=torch.bfloat16, device="cuda")
    y2 = torch.full((A, d), 7.0, dtype=torch.bfloat16, device="cuda")
    abi.moe_expert_ffn_packed_gather(x, k, src, offsets, wgu_p, wd_p, y1, ws)
    assert_ffn_ran_all(ws)
    for _ in range(3):
        abi.moe_expert_ffn_packed_gather(x, k, src, offsets, wgu_p, wd_p, y2, ws_shift)
        assert_ffn_ran_all(ws_shift)
        assert torch.equal(y1.view(torch.int16), y2.view(torch.int16))
        y2.fill_(7.0)


def test_gather_ffn_clamps_K_below_k_like_the_route():
    """A prefix length below k: moe_route raises it to k, and the gathering
    FFN applies the same clamp, so every expert the re-route selected is
    evaluated (bitwise the result with K = k)."""
    T, E, k, d, m = 256, 32, 8, 512, 256
    sh = I.LayerShape(d=d, E=E, m=m, k=k, dtype="bf16")
    prm = I.layer_params(sh, seed=41)
    lg = dev(I.synthetic_rows(T, E, "f32", seed=42), torch.float32)
    A = T * k
    wgu, wd = dev(prm["w_gate_up"], torch.bfloat16), dev(prm["w_down"], torch.bfloat16)
    wgu_p, wd_p = torch.empty_like(wgu), torch.empty_like(wd)
    abi.moe_pack_expert_weights(wgu, wgu_p)
    abi.moe_pack_expert_weights(wd, wd_p)
    x = dev(I.synthetic_rows(T, d, "bf16", seed=43), torch.bfloat16)
    ws = torch.empty(abi.moe_workspace_size(T, E, k, d, m, 1), dtype=torch.uint8, device="cuda")
    ys = {}
    for K in (3, k):
        K_dev = dev(np.array([K], np.int32))
        idx, w = i32((T, k)), f32((T, k))
        abi.moe_route(None, None, None, k, lg, idx, w, K_dev=K_dev)
        assert int(host(idx).max()) == k - 1  # the route selected all of [0, k)
        counts, offsets, src, ros = i32((E,)), i32((E + 1,)), i32((A,)), i32((A,))
        abi.moe_dispatch(idx, E, None, counts, offsets, src, ros, None, ws)
        y = torch.full((A, d), 7.0, dtype=torch.bfloat16, device="cuda")
        abi.moe_expert_ffn_packed_gather(x, k, src, offsets, wgu_p, wd_p, y, ws, K_dev=K_dev)
        assert_ffn_ran_all(ws)
        ys[K] = y
    assert torch.equal(ys[3].view(torch.int16), ys[k].view(torch.int16))
    assert not (host(ys[3]) == 7.0).all(axis=1).any()  # every row written


def test_packed_ffn_per_segment_K_uses_the_largest():
    """K_dev with one K per segment: experts below the largest K are
    evaluated (the same result as that K alone), none above it."""
    E, d, m = 12, 512, 256
    sh = I.LayerShape(d=d, E=E, m=m, k=1, dtype="bf16")
    prm = I.layer_params(sh, seed=9)
    counts = np.array([40, 0, 70, 5, 130, 9, 1, 33, 0, 64, 2, 17], np.int64)
    rows = int(counts.sum())
    offsets = dev(np.concatenate([[0], np.cumsum(counts)]).astype(np.int32))
    xp = dev(I.synthetic_rows(rows, d, "bf16", seed=10), torch.bfloat16)
    wgu, wd = dev(prm["w_gate_up"], torch.bfloat16), dev(prm["w_down"], torch.bfloat16)
    wgu_p, wd_p = torch.empty_like(wgu), torch.empty_like(wd)
    abi.moe_pack_expert_weights(wgu, wgu_p)
    abi.moe_pack_expert_weights(wd, wd_p)
    ws = torch.empty(abi.moe_workspace_size(rows, E, 1, d, m, 3), dtype=torch.uint8, device="cuda")
    y_seg = torch.full((rows, d), 7.0, dtype=torch.bfloat16, device="cuda")
    y_one = torch.full((rows, d), 7.0, dtype=torch.bfloat16, device="cuda")
    abi.moe_expert_ffn_packed(xp, offsets, wgu_p, wd_p, y_seg, ws, K_dev=dev(np.array([2, 7, 3], np.int32)))
    abi.moe_expert_ffn_packed(xp, offsets, wgu_p, wd_p, y_one, ws, K_dev=dev(np.array([7], np.int32)))
    torch.cuda.synchronize()
    assert torch.equal(y_seg.view(torch.int16), y_one.view(torch.int16))
    past = int(np.cumsum(counts)[6])  # rows of experts >= 7 are left unwritten
    assert (host(y_seg)[past:] == 7.0).all()
    assert not (host(y_seg)[:past] == 7.0).all(axis=1).any()


@pytest.mark.parametrize("T,E,k,d,m", [(512, 128, 8, 2048, 768), (4096, 128, 8, 2048, 768),
                                       (37, 6, 3, 512, 256)])
def test_packed_ffn_two_launch_fallback_matches_persistent(T, E, k, d, m, monkeypatch):
    """The one-launch-per-GEMM path (used where the XCD count is unknown)
    gives bitwise the persistent kernel's result."""
    sh = I.LayerShape(d=d, E=E, m=m, k=k, dtype="bf16")
    prm = I.layer_params(sh, seed=2)
    idx, _ = I.synthetic_routing(T, E, k, seed=T + 1)
    x = dev(I.synthetic_rows(T, d, "bf16", seed=T + 2), torch.bfloat16)
    A = T * k
    counts, offsets, src, ros = i32((E,)), i32((E + 1,)), i32((A,)), i32((A,))
    ws = torch.empty(abi.moe_workspace_size(T, E, k, d, m, 1), dtype=torch.uint8, device="cuda")
    abi.moe_dispatch(dev(idx), E, None, counts, offsets, src, ros, None, ws)
    wgu, wd = dev(prm["w_gate_up"], torch.bfloat16), dev(prm["w_down"], torch.bfloat16)
    wgu_p, wd_p = torch.empty_like(wgu), torch.empty_like(wd)
    abi.moe_pack_expert_weights(wgu, wgu_p)
    abi.moe_pack_expert_weights(wd, wd_p)
    y1 = torch.full((A, d), 7.0, dtype=torch.bfloat16, device="cuda")
    y2 = torch.full((A, d), 7.0, dtype=torch.bfloat16, device="cuda")
    abi.moe_expert_ffn_packed_gather(x, k, src, offsets, wgu_p, wd_p, y1, ws)
    assert assert_ffn_ran_all(ws)[0] == abi.FFN_PATH_PERSISTENT
    monkeypatch.setenv("DECOMOE_FFN_TWO_LAUNCH", "1")
    abi.moe_expert_ffn_packed_gather(x, k, src, offsets, wgu_p, wd_p, y2, ws)
    assert assert_ffn_ran_all(ws)[0] == abi.FFN_PATH_TWO_LAUNCH
    monkeypatch.delenv("DECOMOE_FFN_TWO_LAUNCH")
    assert torch.equal(y1.view(torch.int16), y2.view(torch.int16))


# 128-row tiles at 4096 and 1024 tokens, 64-row tiles at 512, 64-row tiles
# streaming the weights at 64
@pytest.mark.parametrize("T", [4096, 1024, 512, 64])
def test_persistent_ffn_repeated_calls_bitwise(T, monkeypatch):
    """Back-to-back persistent calls on one workspace (its counters cleared
    and reused every call) keep giving the two-launch path's bits: each of
    40 calls is compared with it."""
    E, k, d, m = 128, 8, 2048, 768
    sh = I.LayerShape(d=d, E=E, m=m, k=k, dtype="bf16")
    prm = I.layer_params(sh, seed=4)
    idx, _ = I.synthetic_routing(T, E, k, seed=T + 9)
    x = dev(I.synthetic_rows(T, d, "bf16", seed=T + 8), torch.bfloat16)
    A = T * k
    counts, offsets, src, ros = i32((E,)), i32((E + 1,)), i32((A,)), i32((A,))
    ws = torch.empty(abi.moe_workspace_size(T, E, k, d, m, 1), dtype=torch.uint8, device="cuda")
    abi.moe_dispatch(dev(idx), E, None, counts, offsets, src, ros, None, ws)
    wgu, wd = dev(prm["w_gate_up"], torch.bfloat16), dev(prm["w_down"], torch.bfloat16)
    wgu_p, wd_p = torch.empty_like(wgu), torch.empty_like(wd)
    abi.moe_pack_expert_weights(wgu, wgu_p)
    abi.moe_pack_expert_weights(wd, wd_p)
    ref = torch.empty((A, d), dtype=torch.bfloat16, device="cuda")
    monkeypatch.setenv("DECOMOE_FFN_TWO_LAUNCH", "1")
    abi.moe_expert_ffn_packed_gather(x, k, src, offsets, wgu_p, wd_p, ref, ws)
    torch.cuda.synchronize()
    monkeypatch.delenv("DECOMOE_FFN_TWO_LAUNCH")
    ys = [torch.empty((A, d), dtype=torch.bfloat16, device="cuda") for _ in range(4)]
    st = torch.full((40, 4), -1, dtype=torch.int32, device="cuda")
    for i in range(40):
        abi.moe_expert_ffn_packed_gather(x, k, src, offsets, wgu_p, wd_p, ys[i % 4], ws)
        abi.moe_ffn_status(ws, st[i])  # no host wait between the calls
        if i % 4 == 3:
            torch.cuda.synchronize()
            for y in ys:
                assert torch.equal(y.view(torch.int16), ref.view(torch.int16)), i
                y.fill_(7.0)
    s_h = host(st)
    assert (s_h[:, 0] == 0).all() and (s_h[:, 3] == abi.FFN_PATH_PERSISTENT).all()
    assert (s_h[:, 1] == s_h[:, 2]).all() and (s_h[:, 2] == s_h[0, 2]).all() and s_h[0, 2] > 0


def test_expert_ffn_packed_gather_out_of_range_rows_read_token_zero():
    T, E, k, d, m = 64, 4, 2, 512, 256
    sh = I.LayerShape(d=d, E=E, m=m, k=k, dtype="bf16")
    prm = I.layer_params(sh, seed=5)
    idx, _ = I.synthetic_routing(T, E, k, seed=6)
    x = dev(I.synthetic_rows(T, d, "bf16", seed=7), torch.bfloat16)
    A = T * k
    counts, offsets, src, ros = i32((E,)), i32((E + 1,)), i32((A,)), i32((A,))
    ws = torch.empty(abi.moe_workspace_size(T, E, k, d, m, 1), dtype=torch.uint8, device="cuda")
    abi.moe_dispatch(dev(idx), E, None, counts, offsets, src, ros, None, ws)
    bad = torch.tensor([3, 40, 77], dtype=torch.long, device="cuda")
    src[bad] = torch.tensor([-5, A, A + 1000], dtype=torch.int32, device="cuda")
    wgu, wd = dev(prm["w_gate_up"], torch.bfloat16), dev(prm["w_down"], torch.bfloat16)
    wgu_p, wd_p = torch.empty_like(wgu), torch.empty_like(wd)
    abi.moe_pack_expert_weights(wgu, wgu_p)
    abi.moe_pack_expert_weights(wd, wd_p)
    y = torch.empty((A, d), dtype=torch.bfloat16, device="cuda")
    abi.moe_expert_ffn_packed_gather(x, k, src, offsets, wgu_p, wd_p, y, ws)
    # the row-copy path on the rows the gather reads (token 0 for bad entries)
    s_h = host(src).astype(np.int64) // k
    s_h[(s_h < 0) | (s_h >= T)] = 0
    xp = x[torch.as_tensor(s_h, device="cuda")].contiguous()
    y_ref = torch.empty_like(y)
    abi.moe_expert_ffn_packed(xp, offsets, wgu_p, wd_p, y_ref, ws)
    assert torch.equal(y.view(torch.int16), y_ref.view(torch.int16))


# ---------------------------------------------------------------------------
# moe_combine
# ---------------------------------------------------------------------------
# (20000, 2, 2048) and (9000, 4, 2048, f32) write more than 64 MiB: the
# output stores bypass the caches
@pytest.mark.parametrize("T,k,d,dt", [(512, 2, 256, "f32"), (4096, 8, 2048, "bf16"), (1, 8, 2048, "bf16"),
                                      (33, 3, 10, "f32"), (50, 4, 6, "bf16"), (20000, 2, 2048, "bf16"),
                                      (9000, 1, 2048, "f32")])
def test_combine(T, k, d, dt):
    A = T * k
    y = I.synthetic_rows(A, d, dt, seed=A + d)
    ros = I.synthetic_permutation(A, seed=A)
    _, w = I.synthetic_routing(T, max(k, 8), k, seed=T)
    out = torch.empty((T, d), dtype=TDT[dt], device="cuda")
    abi.moe_combine(dev(y, TDT[dt]), dev(ros), dev(w), out)
    ref = oracle.combine(y, ros, w)
    assert rel_inf(host(out), ref) <= TOL[dt]
    assert row_rel(host(out), ref) <= TOL[dt]


@pytest.mark.parametrize("T,E,k,d", [(4096, 128, 8, 2048), (77, 16, 2, 256), (20000, 128, 2, 2048)])
def test_combine_inverts_dispatch(T, E, k, d):
    """Identity experts with unit weights give k*x exactly (k a power of two,
    sums of k bf16 copies exact in float32)."""
    idx, _ = I.synthetic_routing(T, E, k, seed=5)
    x = I.synthetic_rows(T, d, "bf16", seed=6)
    A = T * k
    counts, offsets, src, ros = i32((E,)), i32((E + 1,)), i32((A,)), i32((A,))
    xp = torch.empty((A, d), dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(abi.moe_workspace_size(T, E, k, d, 64, 1), dtype=torch.uint8, device="cuda")
    abi.moe_dispatch(dev(idx), E, dev(x, torch.bfloat16), counts, offsets, src, ros, xp, ws)
    out = torch.empty((T, d), dtype=torch.bfloat16, device="cuda")
    abi.moe_combine(xp, ros, dev(np.ones((T, k), np.float32)), out)
    np.testing.assert_array_equal(host(out), k * x)
