"""Dense-span and RCEP-span MoE layers composed from the C-ABI calls.

Everything computed here runs in libdecomoe.so; this module only owns device
buffers (torch tensors used as plain device memory) and issues the calls in
the order of Algorithm 2 of the paper:

  dense span (before the visual exit):
      moe_route(x) -> moe_dispatch -> moe_expert_ffn -> moe_combine
      (bf16 layers: moe_route_packed and moe_expert_ffn_packed_gather on
      router and expert weights packed at load time; the dispatch then only
      groups the assignments and the expert GEMM reads the token rows)
  RCEP span (from the visual exit on):
      moe_route(x) [full pool] -> moe_calibrate_prefix [s, K]
      -> moe_route(logits, K) [prefix re-route] -> moe_dispatch
      -> moe_expert_ffn(K) -> moe_combine
      (one invocation: moe_calibrate_route_prefix does s, K and the
      re-route in one call; on packed weights moe_route_rcep does the
      routing through the grouping, and with a residual moe_rcep_layer does
      the whole layer)

All calls are asynchronous on one stream and K never leaves the device.
"""

from __future__ import annotations

import numpy as np
import torch

from . import abi

_TORCH_DT = {"f32": torch.float32, "bf16": torch.bfloat16}


def to_device(a: np.ndarray | None, dtype: torch.dtype, device="cuda"):
    """Upload a float32 numpy array (bf16 layers: values already bf16-exact)."""
    if a is None:
        return None
    return torch.from_numpy(np.ascontiguousarray(a)).to(device).to(dtype).contiguous()


def apply_order(params: dict, order: np.ndarray) -> dict:
    """Physical expert reorder (Sec. 3.3 after Eq. 9; Algorithm 1): new
    expert j is native expert order[j] in the router columns, the bias, and
    the gate/up and down tensors.  Done once on the host when the layer is
    loaded: it moves storage and computes nothing."""
    order = np.asarray(order)
    return dict(
        w_r=np.ascontiguousarray(params["w_r"][:, order]),
        bias=None if params["bias"] is None else np.ascontiguousarray(params["bias"][order]),
        w_gate_up=np.ascontiguousarray(params["w_gate_up"][order]),
        w_down=np.ascontiguousarray(params["w_down"][order]),
    )


def calibrate_order_router(x_text: torch.Tensor, w_r: np.ndarray, bias, k: int,
                           seg_offsets=None) -> np.ndarray:
    """Mean-Mass order (Eqs. 8, 9) of one layer from the full-pool routing
    of calibration text rows on the native-order router; each segment is
    one calibration case.  Only the router weights are needed."""
    T = x_text.shape[0]
    E = w_r.shape[1]
    n_seg = 1 if seg_offsets is None else seg_offsets.numel() - 1
    dev = x_text.device
    logits = torch.empty((T, E), dtype=torch.float32, device=dev)
    idx = torch.empty((T, k), dtype=torch.int32, device=dev)
    w = torch.empty((T, k), dtype=torch.float32, device=dev)
    mass = torch.empty((n_seg, E), dtype=torch.float64, device=dev)
    order = torch.empty((E,), dtype=torch.int32, device=dev)
    ws = torch.empty(abi.moe_workspace_size(T, E, k, x_text.shape[1], 1, n_seg), dtype=torch.uint8,
                     device=dev)
    abi.moe_route(x_text, to_device(w_r, torch.float32, dev), to_device(bias, torch.float32, dev), k,
                  logits, idx, w, ws=ws)
    abi.moe_calibrate_prefix(idx, w, E, 1.0, mass, ws, order=order, seg_offsets=seg_offsets)
    return order.cpu().numpy()


class Buffers:
    """Device buffers of one invocation size (T tokens, n_seg segments)."""

    def __init__(self, T: int, d: int, E: int, m: int, k: int, dt: torch.dtype, n_seg: int = 1,
                 device="cuda", x_perm: bool = True):
        i32, f32 = torch.int32, torch.float32
        A = T * k
        self.T, self.n_seg = T, n_seg
        self.logits = torch.empty((T, E), dtype=f32, device=device)
        self.idx_full = torch.empty((T, k), dtype=i32, device=device)
        self.w_full = torch.empty((T, k), dtype=f32, device=device)
        self.mass = torch.empty((n_seg, E), dtype=torch.float64, device=device)
        self.K = torch.empty((n_seg,), dtype=i32, device=device)
        self.idx = torch.empty((T, k), dtype=i32, device=device)
        self.w = torch.empty((T, k), dtype=f32, device=device)
        self.counts = torch.empty((E,), dtype=i32, device=device)
        self.offsets = torch.empty((E + 1,), dtype=i32, device=device)
        self.src_of_row = torch.empty((A,), dtype=i32, device=device)
        self.row_of_slot = torch.empty((A,), dtype=i32, device=device)
        # dispatched token rows; layers on packed weights gather them inside
        # the expert GEMM and need none
        self.x_perm = torch.empty((A, d), dtype=dt, device=device) if x_perm else None
        self.y_perm = torch.empty((A, d), dtype=dt, device=device)
        self.out = torch.empty((T, d), dtype=dt, device=device)
        nbytes = abi.moe_workspace_size(T, E, k, d, m, n_seg)
        self.ws = torch.empty((nbytes,), dtype=torch.uint8, device=device)


class MoELayer:
    """One MoE layer's parameters on the device, in reordered expert order."""

    def __init__(self, params: dict, k: int, dtype: str, device="cuda"):
        dt = _TORCH_DT[dtype]
        self._setup(to_device(params["w_r"], torch.float32, device),
                    to_device(params["bias"], torch.float32, device),
                    to_device(params["w_gate_up"], dt, device), to_device(params["w_down"], dt, device),
                    k, dtype, device)

    @classmethod
    def from_native(cls, w_r: np.ndarray, bias, w_gate_up: torch.Tensor, w_down: torch.Tensor,
                    order, k: int, dtype: str, device="cuda") -> "MoELayer":
        """Load a layer whose expert weights are already on the device in
        native order: the Mean-Mass order (Eq. 9) is applied on the device
        (moe_permute_experts) and the weights are then packed.  The native
        weight tensors are consumed (reused as the packed storage)."""
        self = cls.__new__(cls)
        o = torch.as_tensor(np.asarray(order), dtype=torch.int32).to(device)
        w_r_n = to_device(w_r, torch.float32, device)
        b_n = to_device(bias, torch.float32, device)
        w_r_p = torch.empty_like(w_r_n)
        b_p = torch.empty_like(b_n) if b_n is not None else None
        gu = torch.empty_like(w_gate_up)
        dn = torch.empty_like(w_down)
        abi.moe_permute_experts(o, w_r_n, b_n, w_gate_up, w_down, w_r_p, b_p, gu, dn)
        self._setup(w_r_p, b_p, gu, dn, k, dtype, device, spare=(w_gate_up, w_down))
        return self

    def _setup(self, w_r, bias, w_gate_up, w_down, k, dtype, device, spare=None):
        self.dt = _TORCH_DT[dtype]
        self.k = k
        self.d, self.E = w_r.shape
        self.m = w_down.shape[2]
        self.w_r, self.bias = w_r, bias
        self.w_gate_up, self.w_down = w_gate_up, w_down
        # bf16 layers keep the expert weights in the packed fragment layout
        # (moe_pack_expert_weights), re-laid out once here like the reorder
        self.packed = self.dt == torch.bfloat16 and self.m % 256 == 0 and self.d % 256 == 0
        if self.packed:
            wgu, wd = spare if spare is not None else (torch.empty_like(w_gate_up),
                                                       torch.empty_like(w_down))
            abi.moe_pack_expert_weights(self.w_gate_up, wgu)
            abi.moe_pack_expert_weights(self.w_down, wd)
            self.w_gate_up, self.w_down = wgu, wd
        # bf16 layers with 32-expert blocks route on bf16 MFMA with the
        # router weights split in three bf16 terms (moe_pack_router)
        self.w_r_packed = None
        if self.dt == torch.bfloat16 and self.E % 32 == 0 and self.d % 64 == 0:
            self.w_r_packed = torch.empty((3 * self.d * self.E,), dtype=torch.bfloat16, device=device)
            abi.moe_pack_router(self.w_r, self.w_r_packed)
        self.device = device
        self._bufs: dict = {}
        self._kdev: dict = {}  # device copies of fixed prefix lengths

    def _check_guard(self, guard):
        # predicated calls exist for the packed bf16 path (the stacks that
        # capture Algorithm 2's prefill as one graph)
        if guard is not None and not (self.packed and self.w_r_packed is not None):
            raise ValueError("predicated layers need packed bf16 router and expert weights")

    def _route(self, x, b: Buffers, idx, w, stream=None, guard=None):
        """Router logits into b.logits and the full-pool Top-k."""
        if guard is not None:
            abi.moe_route_packed_if(x, self.w_r_packed, self.bias, self.k, b.logits, idx, w, guard, ws=b.ws,
                                    stream=stream)
        elif self.w_r_packed is not None:
            abi.moe_route_packed(x, self.w_r_packed, self.bias, self.k, b.logits, idx, w, ws=b.ws,
                                 stream=stream)
        else:
            abi.moe_route(x, self.w_r, self.bias, self.k, b.logits, idx, w, ws=b.ws, stream=stream)

    @property
    def one_call(self) -> bool:
        """Packed weights of the shapes the one-call layers take
        (moe_dense_layer, moe_rcep_layer)."""
        return self.packed and self.w_r_packed is not None and self.k <= 32

    def buffers(self, T: int, n_seg: int = 1) -> Buffers:
        key = (T, n_seg)
        if key not in self._bufs:
            self._bufs[key] = Buffers(T, self.d, self.E, self.m, self.k, self.dt, n_seg, self.device,
                                      x_perm=not self.packed)
        return self._bufs[key]

    # -- stages ------------------------------------------------------------
    # `mark`, if given, is called after each ABI call (e.g. to record events).
    # With `residual`, the combine writes out = residual + MoE(x) into `out`
    # (default b.out); `out` may be `residual` itself (in-place hidden state).
    def _experts(self, x, b: Buffers, idx, w, K_dev=None, stream=None, mark=None, residual=None,
                 out=None, guard=None, dispatched=False):
        """dispatch -> expert FFN -> combine; ``dispatched``: the grouping is
        already in b (moe_route_rcep did it)."""
        mark = mark or (lambda: None)
        if guard is not None:
            # the same calls, each run only while the predicate holds
            if not dispatched:
                abi.moe_dispatch_if(idx, self.E, None, b.counts, b.offsets, b.src_of_row, b.row_of_slot, None,
                                    b.ws, guard, stream=stream)
            abi.moe_expert_ffn_packed_gather_if(x, idx.shape[1], b.src_of_row, b.offsets, self.w_gate_up,
                                                self.w_down, b.y_perm, b.ws, guard, K_dev=K_dev,
                                                stream=stream)
            if residual is None:
                raise ValueError("predicated layers combine with the residual")
            abi.moe_combine_residual_if(b.y_perm, b.row_of_slot, w, residual,
                                        b.out if out is None else out, guard, stream=stream)
            return
        if self.packed:
            # the expert GEMM reads the token rows through src_of_row: the
            # dispatch only groups the assignments
            if not dispatched:
                abi.moe_dispatch(idx, self.E, None, b.counts, b.offsets, b.src_of_row, b.row_of_slot,
                                 None, b.ws, stream=stream)
                mark()
            abi.moe_expert_ffn_packed_gather(x, idx.shape[1], b.src_of_row, b.offsets, self.w_gate_up,
                                             self.w_down, b.y_perm, b.ws, K_dev=K_dev, stream=stream)
        else:
            abi.moe_dispatch(idx, self.E, x, b.counts, b.offsets, b.src_of_row, b.row_of_slot,
                             b.x_perm, b.ws, stream=stream)
            mark()
            abi.moe_expert_ffn(b.x_perm, b.offsets, self.w_gate_up, self.w_down, b.y_perm, b.ws,
                               K_dev=K_dev, stream=stream)
        mark()
        out = b.out if out is None else out
        if residual is None:
            abi.moe_combine(b.y_perm, b.row_of_slot, w, out, stream=stream)
        else:
            abi.moe_combine_residual(b.y_perm, b.row_of_slot, w, residual, out, stream=stream)
        mark()

    def forward_dense(self, x: torch.Tensor, b: Buffers | None = None, stream=None,
                      mark=None, residual=None, out=None, guard=None) -> Buffers:
        """Full expert pool (layers before the visual exit).  ``guard`` =
        (int32 device tensor g, lo, hi): every call runs only while
        lo <= g[0] < hi (packed layers, with a residual)."""
        self._check_guard(guard)
        b = b or self.buffers(x.shape[0])
        if self.one_call and mark is None and guard is None:
            # the whole layer in one call (the dispatch also clears the
            # expert FFN's counters)
            abi.moe_dense_layer(x, self.w_r_packed, self.bias, self.k, self.w_gate_up, self.w_down, residual,
                                b.out if out is None else out, b.logits, b.idx, b.w, b.counts, b.offsets,
                                b.src_of_row, b.row_of_slot, b.y_perm, b.ws, stream=stream)
            return b
        self._route(x, b, b.idx, b.w, stream=stream, guard=guard)
        if mark:
            mark()
        self._experts(x, b, b.idx, b.w, stream=stream, mark=mark, residual=residual, out=out, guard=guard)
        return b

    def prefix_tensor(self, K: int) -> torch.Tensor:
        """A device copy of a host prefix length, checked against Eq. 12's
        range k <= K <= E (made once per value and kept, so that a captured
        graph can read it)."""
        K = int(K)
        if not self.k <= K <= self.E:
            raise ValueError(f"prefix length {K} outside [k, E] = [{self.k}, {self.E}]")
        if K not in self._kdev:
            self._kdev[K] = torch.full((4,), K, dtype=torch.int32, device=self.device)[:1]
        return self._kdev[K]

    def forward_prefix(self, x: torch.Tensor, K, b: Buffers | None = None,
                       stream=None, mark=None, residual=None, out=None) -> Buffers:
        """A given prefix length instead of Eq. 12 (the fixed-prefix variant
        of the component ablation, Table 2): logits over all E experts, Top-k
        inside [0, K), experts [0, K) only.  K is a host int (checked:
        k <= K <= E) or a device int32 tensor holding K (the route and the
        gathering expert FFN both raise a value below k to k)."""
        K_dev = K if isinstance(K, torch.Tensor) else self.prefix_tensor(K)
        b = b or self.buffers(x.shape[0])
        if self.w_r_packed is not None:
            abi.moe_route_packed(x, self.w_r_packed, self.bias, self.k, b.logits, b.idx, b.w, K_dev=K_dev,
                                 ws=b.ws, stream=stream)
        else:
            abi.moe_route(x, self.w_r, self.bias, self.k, b.logits, b.idx, b.w, K_dev=K_dev, ws=b.ws,
                          stream=stream)
        if mark:
            mark()
        self._experts(x, b, b.idx, b.w, K_dev=K_dev, stream=stream, mark=mark, residual=residual, out=out)
        return b

    def forward_rcep_chained(self, h: torch.Tensor, p: float, b: Buffers, chained: bool, stream=None,
                             K_out=None) -> Buffers:
        """One RCEP layer of a stack whose combines are chained
        (moe_rcep_layer_chained): with ``chained`` the previous layer's
        combine with the residual (its y_perm, row_of_slot and re-routed
        weights, left in ``b``) first updates h in place; then this layer's
        routing and expert FFN over h.  Its own combine is left in ``b`` for
        the next chained layer or for moe_combine_residual."""
        if not self.one_call:
            raise ValueError("chained layers need packed bf16 weights")
        K = b.K if K_out is None else K_out
        prev = (b.y_perm, b.row_of_slot, b.w) if chained else None
        abi.moe_rcep_layer_chained(prev, h, self.w_r_packed, self.bias, self.k, p, self.w_gate_up, self.w_down,
                                   b.logits, b.idx_full, b.w_full, b.mass, K, b.idx, b.w, b.counts, b.offsets,
                                   b.src_of_row, b.row_of_slot, b.y_perm, b.ws, stream=stream)
        return b

    def forward_rcep(self, x: torch.Tensor, p: float, seg_offsets=None, b: Buffers | None = None,
                     stream=None, mark=None, residual=None, out=None, K_out=None, guard=None) -> Buffers:
        """Prefix-restricted layer (from the visual exit on, Algorithm 2).
        K_out ([n_seg] int32, default b.K) receives the prefix lengths.
        ``guard``: as in forward_dense (one invocation only)."""
        self._check_guard(guard)
        n_seg = 1 if seg_offsets is None else seg_offsets.numel() - 1
        b = b or self.buffers(x.shape[0], n_seg)
        K = b.K if K_out is None else K_out
        mk = mark or (lambda: None)
        if seg_offsets is None and self.one_call and mark is None:
            # one invocation on packed weights: the whole layer in one call
            # (its routing launch also clears the expert FFN's counters)
            abi.moe_rcep_layer(x, self.w_r_packed, self.bias, self.k, p, self.w_gate_up, self.w_down, residual,
                               b.out if out is None else out, b.logits, b.idx_full, b.w_full, b.mass, K, b.idx,
                               b.w, b.counts, b.offsets, b.src_of_row, b.row_of_slot, b.y_perm, b.ws,
                               guard=guard, stream=stream)
            return b
        if seg_offsets is None and self.packed and self.w_r_packed is not None:
            # one invocation on packed weights: routing, masses, K, the
            # prefix re-route and the grouping in one call
            abi.moe_route_rcep(x, self.w_r_packed, self.bias, self.k, p, b.logits, b.idx_full, b.w_full, b.mass,
                               K, b.idx, b.w, b.counts, b.offsets, b.src_of_row, b.row_of_slot, b.ws,
                               guard=guard, stream=stream)
            mk()
            self._experts(x, b, b.idx, b.w, K_dev=K, stream=stream, mark=mark, residual=residual, out=out,
                          guard=guard, dispatched=True)
            return b
        if guard is not None:
            raise ValueError("predicated RCEP layers take one invocation on packed weights")
        self._route(x, b, b.idx_full, b.w_full, stream=stream)
        mk()
        if seg_offsets is None:
            # one invocation: masses, K and the prefix re-route in one call
            abi.moe_calibrate_route_prefix(b.logits, b.idx_full, b.w_full, p, b.mass, K, b.idx, b.w,
                                           stream=stream)
        else:
            abi.moe_calibrate_prefix(b.idx_full, b.w_full, self.E, p, b.mass, b.ws, K_out=K,
                                     seg_offsets=seg_offsets, stream=stream)
            abi.moe_route(None, None, None, self.k, b.logits, b.idx, b.w, seg_offsets=seg_offsets,
                          K_dev=K, stream=stream)
        mk()
        self._experts(x, b, b.idx, b.w, K_dev=K, stream=stream, mark=mark, residual=residual,
                      out=out)
        return b
