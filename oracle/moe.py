"""Plain, slow, fp64 CPU oracle of the RCEP MoE layer of DecoMoE.

TEST INFRASTRUCTURE ONLY: used by tests/, by the smoke check and by the
bench's ``cpu_baseline`` leg; never by the product path.  It shares no code
with the HIP path and imports nothing from it.

Every function below follows one passage of the paper and says which.  All
arithmetic is numpy float64 on exactly widened inputs (bf16 and fp32 values
widen to fp64 without rounding); there is no blocking, fusion or reordering
beyond what the cited definition states.

Notation (paper, Sec. 3.1 and Sec. 3.3):
  x      token rows of one MoE invocation, shape [T, d]
  W_r    router weights, [d, E] (logits a = x W_r + b)
  a      router logits [T, E];  q = softmax(a) over all E experts (Eq. 1)
  R_i    full-pool Top-k expert set of token i (Eq. 10)
  s_e    activated mass of expert e over an invocation (Eq. 11)
  M_e    text-token routed mass of expert e for one calibration case (Eq. 8)
  pi     Mean-Mass expert order (Eq. 9)
  K      retained prefix length, max(k, K_hat) (Eq. 12)

Readings of points the paper leaves open are marked READING and are listed
with their justification in the design notes of the repository.

Parity status: every function is pinned by the CPU tests in
tests/test_oracle_*.py (brute force on tiny inputs, closed forms, invariants,
hand-worked examples).  No function is "parity unpinned".
"""

from __future__ import annotations

import numpy as np

F64 = np.float64

__all__ = [
    "router_logits",
    "softmax",
    "topk_by_logit",
    "renormalised_topk_weights",
    "full_pool_route",
    "prefix_route",
    "activated_mass",
    "routed_mass",
    "mean_mass_order",
    "permute_experts",
    "prefix_length",
    "dispatch",
    "silu",
    "expert_ffn_rows",
    "combine",
    "drop_visual_block",
    "moe_layer_dense",
    "moe_layer_rcep",
    "moe_stack",
    "savb_gate_feature",
    "savb_gate",
    "segment_of_tokens",
]


# --------------------------------------------------------------------------
# Router (Sec. 3.1, Eq. 1)
# --------------------------------------------------------------------------
def router_logits(x, w_r, bias=None):
    """Router logits a_i = x_i W_r (+ b) over all E experts.

    Eq. 1 defines the router probability as a softmax of these logits.  The
    bias term is an addition of this workload's synthetic router (READING:
    the paper's router has no bias; a zero bias gives the paper's form).
    """
    a = np.asarray(x, F64) @ np.asarray(w_r, F64)
    if bias is not None:
        a = a + np.asarray(bias, F64)[None, :]
    return a


def softmax(a):
    """Row-wise softmax over the last axis (Eq. 1), the literal definition."""
    a = np.asarray(a, F64)
    z = np.exp(a - a.max(axis=-1, keepdims=True))
    return z / z.sum(axis=-1, keepdims=True)


def topk_by_logit(a, k):
    """TopK of Eqs. 7 and 10: the k experts with the largest probability.

    Softmax is strictly increasing in each logit, so in exact arithmetic the
    Top-k of q = softmax(a) is the Top-k of a.  The selection is done on the
    logits, which are exact inputs here (READING: equal logits go to the
    lower expert index; slots are stored by descending logit).
    """
    a = np.asarray(a, F64)
    T, E = a.shape
    if not 1 <= k <= E:
        raise ValueError("k must lie in [1, E]")
    # stable argsort of -a: equal keys keep ascending expert index
    order = np.argsort(-a, axis=1, kind="stable")
    return order[:, :k].astype(np.int64)


def renormalised_topk_weights(q, idx):
    """The summand of Eqs. 8 and 11: q_e / sum_{e' in R_i} q_e' for e in R_i."""
    sel = np.take_along_axis(np.asarray(q, F64), idx, axis=1)
    return sel / sel.sum(axis=1, keepdims=True)


def full_pool_route(a, k):
    """Runtime full-pool routing (Eq. 10) with renormalised weights (Eq. 11).

    Returns (idx [T,k], w [T,k]) where w_{i,j} = q_{i,idx} / sum over R_i,
    q being the softmax over all E experts (Eq. 1).  With K = E this is
    also the routing of the dense (unsliced) layer.
    """
    q = softmax(a)
    idx = topk_by_logit(a, k)
    return idx, renormalised_topk_weights(q, idx)


def prefix_route(a, K, k):
    """Prefix-restricted re-route (Sec. 3.3 after Eq. 12; Algorithm 2).

    The logits are restricted to the first K reordered experts, a new
    softmax is taken over that prefix, Top-k is rerun inside it and the
    selected weights are renormalised.  The full-pool Top-k set is not
    intersected with the prefix.  Requires k <= K <= E.
    """
    a = np.asarray(a, F64)
    if not k <= K <= a.shape[1]:
        raise ValueError("need k <= K <= E")
    ap = a[:, :K]
    qt = softmax(ap)
    idx = topk_by_logit(ap, k)
    return idx, renormalised_topk_weights(qt, idx)


# --------------------------------------------------------------------------
# Masses, calibration order and prefix length (Sec. 3.3, Eqs. 8, 9, 11, 12)
# --------------------------------------------------------------------------
def activated_mass(idx, w, E):
    """Activated mass s_e = sum_i 1[e in R_i] w_{i,e} (Eq. 11).

    The sum runs over the tokens of one invocation in ascending token
    order and, within a token, ascending slot order, in fp64.
    """
    idx = np.asarray(idx)
    w = np.asarray(w, F64)
    s = np.zeros(E, F64)
    for i in range(idx.shape[0]):
        for j in range(idx.shape[1]):
            s[idx[i, j]] += w[i, j]
    return s


def routed_mass(idx, w, E):
    """Text-token routed mass of one calibration case (Eq. 8).

    M_e = (1/|T_c|) sum over the case's text tokens of the renormalised
    Top-k weight of e; idx and w hold the rows of those text tokens only.
    An empty case has no defined mean and is rejected.
    """
    n = np.asarray(idx).shape[0]
    if n == 0:
        raise ValueError("a calibration case needs at least one text token")
    return activated_mass(idx, w, E) / n


def mean_mass_order(case_masses):
    """Mean-Mass order pi (Eq. 9): argsort, descending, of the case mean.

    ``case_masses`` is [n_cases, E]; masses are averaged first within a case
    (Eq. 8) and then across cases (App. A.4).  READING: equal means keep the
    lower native index first (a stable sort).  pi[j] is the native index of
    the expert stored at reordered position j.
    """
    cm = np.asarray(case_masses, F64)
    if cm.shape[0] == 0:
        raise ValueError("need at least one calibration case")
    total = np.zeros(cm.shape[1], F64)
    for c in range(cm.shape[0]):  # cases summed in order
        total = total + cm[c]
    mean = total / cm.shape[0]
    return np.argsort(-mean, kind="stable").astype(np.int64), mean


def permute_experts(pi, w_r, bias, w_gate_up, w_down):
    """Apply pi to router outputs and expert tensors (Sec. 3.3 after Eq. 9;
    Algorithm 1): new expert j is native expert pi[j].  Storage changes,
    the function of the unsliced layer does not."""
    pi = np.asarray(pi)
    return (
        np.asarray(w_r)[:, pi],
        None if bias is None else np.asarray(bias)[pi],
        np.asarray(w_gate_up)[pi],
        np.asarray(w_down)[pi],
    )


def prefix_length(s, p, k):
    """Prefix length of Eq. 12: K = max(k, K_hat),
    K_hat = min{K in 1..E : sum_{e<=K} s_e / sum_{e<=E} s_e >= p}.

    READING: the ratio test is taken as c_K >= p * tot in fp64, where c_K is
    the running sum of s in expert order and tot is its last element, so that
    K_hat exists for every p in (0, 1].  An all-zero s (an empty invocation)
    gives K_hat = 1 and hence K = k.
    """
    if not (0.0 < p <= 1.0):
        raise ValueError("p must lie in (0, 1]")
    s = np.asarray(s, F64)
    E = s.shape[0]
    if not 1 <= k <= E:
        raise ValueError("k must lie in [1, E]")
    c = np.zeros(E, F64)
    run = 0.0
    for e in range(E):
        run += s[e]
        c[e] = run
    thr = F64(p) * c[E - 1]
    k_hat = E
    for K in range(1, E + 1):
        if c[K - 1] >= thr:
            k_hat = K
            break
    return max(k, k_hat)


def segment_of_tokens(seg_offsets, T):
    """Invocation (segment) id of every token; one segment when None."""
    if seg_offsets is None:
        return np.zeros(T, np.int64), np.array([0, T], np.int64)
    so = np.asarray(seg_offsets, np.int64)
    seg = np.zeros(T, np.int64)
    for s in range(len(so) - 1):
        seg[so[s]:so[s + 1]] = s
    return seg, so


# --------------------------------------------------------------------------
# Dispatch, expert FFN, combine (Algorithm 2: evaluate and combine only the
# first K physically contiguous expert MLPs)
# --------------------------------------------------------------------------
def dispatch(idx, E):
    """Group the T*k (token, slot) assignments by expert.

    READING: the assignment list in (token, slot) order is sorted stably by
    expert, so within one expert the rows ascend by token.  Returns
    counts [E], offsets [E+1], src_of_row [T*k] (row -> token*k + slot) and
    row_of_slot [T*k] (its inverse).
    """
    idx = np.asarray(idx, np.int64)
    T, k = idx.shape
    keys = idx.reshape(-1)
    src_of_row = np.array(sorted(range(T * k), key=lambda a: keys[a]), np.int64)
    counts = np.bincount(keys, minlength=E).astype(np.int64) if T * k else np.zeros(E, np.int64)
    offsets = np.zeros(E + 1, np.int64)
    offsets[1:] = np.cumsum(counts)
    row_of_slot = np.empty(T * k, np.int64)
    row_of_slot[src_of_row] = np.arange(T * k)
    return counts, offsets, src_of_row, row_of_slot


def silu(z):
    """SiLU(z) = z / (1 + exp(-z))."""
    z = np.asarray(z, F64)
    with np.errstate(over="ignore"):
        return z / (1.0 + np.exp(-z))


def expert_ffn_rows(x_rows, expert_of_row, w_gate_up, w_down):
    """SwiGLU expert MLP per dispatched row (gate, up and down projections,
    App. A.3 Eq. 15 counts them as 6 d m FLOPs per row and expert).

    READING: y = W_down (SiLU(W_gate x) * (W_up x)); the gate and up weights
    of expert e are rows [0, m) and [m, 2m) of w_gate_up[e] ([2m, d]);
    w_down[e] is [d, m].
    """
    x_rows = np.asarray(x_rows, F64)
    R = x_rows.shape[0]
    E, two_m, d = w_gate_up.shape
    m = two_m // 2
    y = np.zeros((R, d), F64)
    expert_of_row = np.asarray(expert_of_row, np.int64)
    for e in np.unique(expert_of_row):
        rows = np.nonzero(expert_of_row == e)[0]
        wgu = np.asarray(w_gate_up[e], F64)
        wd = np.asarray(w_down[e], F64)
        xe = x_rows[rows]
        g = xe @ wgu[:m].T
        u = xe @ wgu[m:].T
        y[rows] = (silu(g) * u) @ wd.T
    return y


def combine(y_rows, row_of_slot, w):
    """Weighted combine: out_i = sum_j w_{i,j} y_{row_of_slot(i,j)}, fp64,
    slots summed in order j = 0..k-1."""
    w = np.asarray(w, F64)
    T, k = w.shape
    y_rows = np.asarray(y_rows, F64)
    d = y_rows.shape[1] if y_rows.ndim == 2 else 0
    out = np.zeros((T, d), F64)
    for j in range(k):
        out += w[:, j:j + 1] * y_rows[np.asarray(row_of_slot)[np.arange(T) * k + j]]
    return out


def drop_visual_block(h, v0, v1):
    """SAVB visual-block removal from the hidden state (Sec. 3.2 after
    Eq. 3; Algorithm 2): the rows [v0, v1) of the contiguous visual block
    are removed and the remaining rows keep their order."""
    h = np.asarray(h)
    S = h.shape[0]
    if not 0 <= v0 <= v1 <= S:
        raise ValueError("need 0 <= v0 <= v1 <= S")
    return np.concatenate([h[:v0], h[v1:]], axis=0)


# --------------------------------------------------------------------------
# One layer (composition of the steps above)
# --------------------------------------------------------------------------
def _experts_and_combine(x, idx, w, w_gate_up, w_down, E):
    counts, offsets, src_of_row, row_of_slot = dispatch(idx, E)
    k = idx.shape[1]
    tok = src_of_row // k
    exp_of_row = np.asarray(idx).reshape(-1)[src_of_row]
    y = expert_ffn_rows(np.asarray(x, F64)[tok], exp_of_row, w_gate_up, w_down)
    out = combine(y, row_of_slot, w)
    return dict(counts=counts, offsets=offsets, src_of_row=src_of_row,
                row_of_slot=row_of_slot, y_rows=y, out=out)


def moe_layer_dense(x, w_r, bias, w_gate_up, w_down, k, logits=None):
    """Dense-span MoE layer (full expert pool; Algorithm 2, layers before
    the visual exit): full-pool Top-k routing, all E experts eligible.

    ``logits`` may be given to teacher-force the routing input.
    """
    a = router_logits(x, w_r, bias) if logits is None else np.asarray(logits, F64)
    E = a.shape[1]
    idx, w = full_pool_route(a, k)
    res = dict(logits=a, idx=idx, w=w)
    res.update(_experts_and_combine(x, idx, w, w_gate_up, w_down, E))
    return res


def moe_layer_rcep(x, w_r, bias, w_gate_up, w_down, k, p, seg_offsets=None,
                   logits=None, K_override=None):
    """RCEP-span MoE layer on reordered parameters (Sec. 3.3; Algorithm 2,
    layers from the visual exit on).

    Per invocation (segment): full-pool Top-k and activated mass (Eqs. 10,
    11), prefix length (Eq. 12), prefix re-route, then only experts [0, K)
    are evaluated and combined.  ``logits`` teacher-forces the routing input;
    ``K_override`` (one K per segment) replaces Eq. 12's result, for
    comparing downstream stages when a near-tie decides K.
    """
    a = router_logits(x, w_r, bias) if logits is None else np.asarray(logits, F64)
    T, E = a.shape
    _, so = segment_of_tokens(seg_offsets, T)
    n_seg = len(so) - 1
    idx_full, w_full = full_pool_route(a, k) if T else (
        np.zeros((0, k), np.int64), np.zeros((0, k), F64))
    mass = np.zeros((n_seg, E), F64)
    K = np.zeros(n_seg, np.int64)
    idx = np.zeros((T, k), np.int64)
    w = np.zeros((T, k), F64)
    for s in range(n_seg):
        lo, hi = so[s], so[s + 1]
        mass[s] = activated_mass(idx_full[lo:hi], w_full[lo:hi], E)
        K[s] = prefix_length(mass[s], p, k) if K_override is None else K_override[s]
        if hi > lo:
            idx[lo:hi], w[lo:hi] = prefix_route(a[lo:hi], int(K[s]), k)
    res = dict(logits=a, idx_full=idx_full, w_full=w_full, mass=mass, K=K,
               idx=idx, w=w)
    res.update(_experts_and_combine(x, idx, w, w_gate_up, w_down, E))
    return res


# --------------------------------------------------------------------------
# A stack of MoE blocks (Algorithm 2's loop over layers)
# --------------------------------------------------------------------------
def moe_stack(h, layers, k, p, exit_layer=None, v0=0, v1=0, seg_offsets=None,
              after_exit="rcep", K_fixed=None):
    """Algorithm 2 over a stack of MoE blocks with the residual stream
    h <- h + MoE_l(h) between blocks (the blocks' attention sublayers are
    not part of this stack).

    ``layers`` holds each layer's reordered parameters (dicts with w_r,
    bias, w_gate_up, w_down).  READING (exit placement): ``exit_layer`` is
    the first text-only layer; the visual rows [v0, v1) are removed at its
    entrance (SAVB, Sec. 3.2), layers before it run the dense span over all
    rows and layers from it on run the RCEP span (Sec. 3.3).  None: no exit,
    every layer dense.  0 with v0 == v1: RCEP in every layer (decode).

    ``after_exit`` selects what the layers from the exit on run, for the
    component ablation (Table 2): "rcep" (the prefix of Eq. 12), "dense"
    (the full expert pool: the visual exit alone) or "fixed" (a given prefix
    length instead of Eq. 12: ``K_fixed``, one int for every such layer or a
    sequence indexed by layer; each must satisfy k <= K <= E).

    Returns the final hidden rows and, per layer, K (None for dense layers).
    """
    if after_exit not in ("rcep", "dense", "fixed"):
        raise ValueError("after_exit is 'rcep', 'dense' or 'fixed'")
    if after_exit == "fixed" and K_fixed is None:
        raise ValueError("the fixed prefix needs K_fixed")
    h = np.asarray(h, F64)
    Ks = []
    for l, prm in enumerate(layers):
        rcep = exit_layer is not None and l >= exit_layer and after_exit != "dense"
        if exit_layer is not None and l == exit_layer:
            h = drop_visual_block(h, v0, v1)
        if rcep:
            K_over = None
            if after_exit == "fixed":
                K_l = int(K_fixed) if np.ndim(K_fixed) == 0 else int(K_fixed[l])
                if not k <= K_l <= np.asarray(prm["w_r"]).shape[1]:
                    raise ValueError("need k <= K_fixed <= E")
                n_seg = 1 if seg_offsets is None else len(seg_offsets) - 1
                K_over = [K_l] * n_seg
            r = moe_layer_rcep(h, prm["w_r"], prm["bias"], prm["w_gate_up"], prm["w_down"], k, p,
                               seg_offsets=seg_offsets, K_override=K_over)
            Ks.append(r["K"])
        else:
            r = moe_layer_dense(h, prm["w_r"], prm["bias"], prm["w_gate_up"], prm["w_down"], k)
            Ks.append(None)
        h = h + r["out"]
    return h, Ks


# --------------------------------------------------------------------------
# SAVB exit gate (Sec. 3.2, Eqs. 2 and 3)
# --------------------------------------------------------------------------
def savb_gate_feature(text_rows):
    """Gate feature of Eq. 2: x = [mean of the first n - 1 text states;
    the final text state], width 2d.

    READING: with a single text token (n = 1) the mean over no rows is the
    zero vector.
    """
    t = np.asarray(text_rows, F64)
    n, d = t.shape
    if n < 1:
        raise ValueError("need at least one text row")
    pooled = t[:n - 1].sum(axis=0) / (n - 1) if n > 1 else np.zeros(d, F64)
    return np.concatenate([pooled, t[n - 1]])


def savb_gate(text_rows, w1, b1, w2, b2, theta):
    """Exit probability and decision of Eq. 3: p_exit = softmax(g(x))_1,
    Exit = 1[p_exit >= theta], for the two-class MLP
    g(x) = W2 act(W1 x + b1) + b2 (hidden width of W1's rows; App. A.3
    counts its two products).

    READING: the hidden activation is ReLU (the paper names the layer sizes,
    not the activation); class 1 is the exit class.
    Returns (p_exit, exit, x, z).
    """
    x = savb_gate_feature(text_rows)
    hid = np.maximum(np.asarray(w1, F64) @ x + np.asarray(b1, F64), 0.0)
    z = np.asarray(w2, F64) @ hid + np.asarray(b2, F64)
    q = softmax(z[None, :])[0]
    p_exit = float(q[1])
    return p_exit, bool(p_exit >= theta), x, z
