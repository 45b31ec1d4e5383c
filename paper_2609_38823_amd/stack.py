"""A stack of MoE blocks on the device: the per-layer loop of Algorithm 2.

Prefill (the 48-layer stack over 7680 visual + 512 text rows):

    layers [0, exit)   dense span over all rows      h <- h + MoE_l(h)
    entrance of exit   drop_visual_block             h <- h[text rows]
    layers [exit, L)   RCEP span over the text rows  h <- h + MoE_l(h)

Decode (64 single text tokens): the RCEP span in every layer, captured once
as a HIP graph and replayed per step.

Gated prefill (``forward_gated``): the SAVB gate (Eqs. 2-3) runs at
candidate layers and its device flag decides the exit layer.

The residual connection is folded into each layer's combine
(moe_combine_residual), so a layer is route -> [calibrate -> re-route] ->
dispatch -> expert FFN -> combine+residual, all in libdecomoe.so, with K
kept on the device per layer (``K_trace``).  The blocks' attention
sublayers are not part of this stack.

Calibration (Eqs. 8, 9): 512 calibration rows enter layer 0 and are carried
through the stack with the full expert pool (dense span), so each layer's
Mean-Mass order comes from the full-pool routing of the calibration rows'
own hidden states at that layer (one calibration case).  The order is
applied on the device (moe_permute_experts) before the weights are packed.
"""

from __future__ import annotations

import numpy as np
import torch

from . import abi, inputs as I
from .layer import Buffers, MoELayer, calibrate_order_router, to_device


class MoEStack:
    """Device-resident stack of ``n_layers`` MoE layers of one workload's shape."""

    def __init__(self, wl: I.Workload, n_layers: int | None = None, calib_rows: int = 512,
                 device="cuda", progress=None):
        sh = wl.shape
        self.wl, self.sh = wl, sh
        self.L = n_layers or wl.layers
        self.device = device
        self.dt = torch.bfloat16 if sh.dtype == "bf16" else torch.float32
        self.layers: list[MoELayer] = []
        self.orders: list[np.ndarray] = []
        self._bufs: dict = {}
        self._h: dict = {}
        # calib_h[l]: the calibration rows entering layer l
        self.calib_h: list[torch.Tensor] = []
        calib = to_device(I.tokens(sh, calib_rows, seed=wl.seed, stream="calib"), self.dt, device)
        for l in range(self.L):
            rp = I.router_params(sh, wl.seed, l)
            self.calib_h.append(calib)
            order = calibrate_order_router(calib, rp["w_r"], rp["bias"], sh.k)
            gu, dn = I.device_expert_weights(sh, wl.seed, l, device)
            layer = MoELayer.from_native(rp["w_r"], rp["bias"], gu, dn, order, sh.k, sh.dtype, device)
            self.layers.append(layer)
            self.orders.append(order)
            del gu, dn
            nxt = torch.empty_like(calib)
            layer.forward_dense(calib, b=self.buffers(calib_rows), residual=calib, out=nxt)
            calib = nxt
            if progress:
                progress(l)
        # row l, column 0: K of layer l when it runs the RCEP span (rows are
        # 16 bytes so that every row is an aligned ABI array)
        self.K_trace = torch.zeros((self.L, 4), dtype=torch.int32, device=device)

    def buffers(self, T: int) -> Buffers:
        """Work buffers for T rows, shared by all layers (one stream)."""
        if T not in self._bufs:
            sh = self.sh
            packed = bool(self.layers) and self.layers[0].packed
            self._bufs[T] = Buffers(T, sh.d, sh.E, sh.m, sh.k, self.dt, 1, self.device, x_perm=not packed)
        return self._bufs[T]

    def hidden(self, T: int, tag: str = "h") -> torch.Tensor:
        key = (T, tag)
        if key not in self._h:
            self._h[key] = torch.empty((T, self.sh.d), dtype=self.dt, device=self.device)
        return self._h[key]

    def layer_forward(self, l: int, src: torch.Tensor, dst: torch.Tensor, rcep: bool, p: float,
                      stream=None, mark=None, K_fixed=None, guard=None) -> Buffers:
        """One block: dst = src + MoE_l(src); dst may be src (in place).
        rcep: the RCEP span (Eq. 12's K, or the prefix length K_fixed when
        given: a host int or a device int32 tensor); else the full expert
        pool.  guard: (int32 device tensor g, lo, hi), the block runs only
        while lo <= g[0] < hi (packed layers)."""
        b = self.buffers(src.shape[0])
        layer = self.layers[l]
        if rcep and K_fixed is not None:
            return layer.forward_prefix(src, K_fixed, b=b, stream=stream, mark=mark, residual=src, out=dst)
        if rcep:
            return layer.forward_rcep(src, p, b=b, stream=stream, mark=mark, residual=src, out=dst,
                                      K_out=self.K_trace[l, :1], guard=guard)
        return layer.forward_dense(src, b=b, stream=stream, mark=mark, residual=src, out=dst, guard=guard)

    def forward(self, x: torch.Tensor, n_visual: int, p: float, exit_layer: int | None,
                stream=None, hook=None, after_exit: str = "rcep", K_fixed=None) -> torch.Tensor:
        """Run the stack over x [T, d] (visual rows [0, n_visual) first).

        exit_layer is the first text-only layer: the visual rows are removed
        at its entrance and it and every later layer run the RCEP span;
        None runs every layer dense.  x itself is not modified.  Returns the
        final hidden rows (a buffer owned by the stack).  ``hook(l, src)``,
        if given, is called before layer l with its input rows.
        after_exit selects the layers from the exit on (component ablation,
        Table 2): "rcep" (Eq. 12), "dense" (all experts: the visual exit
        alone) or "fixed" (the prefix length K_fixed: a host int, checked
        against [k, E], or a device int32 tensor).
        With packed weights and no hook, the RCEP layers are chained
        (moe_rcep_layer_chained): layer l's combine with the residual runs
        inside layer l + 1's first launch, the last one's as
        moe_combine_residual; the results are bitwise those of the separate
        calls.
        """
        if after_exit not in ("rcep", "dense", "fixed"):
            raise ValueError("after_exit is 'rcep', 'dense' or 'fixed'")
        if after_exit == "fixed" and K_fixed is None:
            raise ValueError("the fixed prefix needs K_fixed")
        T = x.shape[0]
        src = x
        h = self.hidden(T)
        chain = hook is None and after_exit == "rcep" and exit_layer is not None and exit_layer < self.L \
            and self.chainable()
        for l in range(self.L):
            if exit_layer is not None and l == exit_layer and n_visual > 0:
                ht = self.hidden(T - n_visual, "text")
                abi.drop_visual_block(src, 0, n_visual, ht, stream=stream)
                src, h = ht, ht
            if hook:
                hook(l, src)
            rcep = exit_layer is not None and l >= exit_layer and after_exit != "dense"
            if chain and rcep:
                if src is x:  # no layer before the exit: the rows are updated in a copy
                    h.copy_(x)
                    src = h
                self.layers[l].forward_rcep_chained(src, p, self.buffers(src.shape[0]), l > exit_layer,
                                                    stream=stream, K_out=self.K_trace[l, :1])
                continue
            dst = h if src is x else src
            self.layer_forward(l, src, dst, rcep, p, stream=stream,
                               K_fixed=K_fixed if after_exit == "fixed" else None)
            src = dst
        if chain:
            b = self.buffers(src.shape[0])
            abi.moe_combine_residual(b.y_perm, b.row_of_slot, b.w, src, src, stream=stream)
        return src

    def forward_gated(self, x: torch.Tensor, n_visual: int, p: float, gates: dict, theta: float,
                      stream=None):
        """Algorithm 2 with the SAVB gate choosing the exit (Sec. 3.2).

        Before each candidate layer l (the keys of ``gates``: per layer a
        dict of device tensors w1, b1, w2, b2) while the visual block is
        still present, moe_savb_gate evaluates Eqs. 2-3 on the text rows.
        Its flag is read on the host once per candidate -- the only host
        wait, since it fixes the row count of the layers that follow; on an
        exit, drop_visual_block_if removes the visual rows and layers l..
        run the RCEP span.  Returns (final rows, exit layer or None,
        [(layer, p_exit)] of the evaluated candidates).
        """
        T = x.shape[0]
        src = x
        h = self.hidden(T)
        d = self.sh.d
        n_text = T - n_visual
        hid = next(iter(gates.values()))["w1"].shape[0] if gates else 1
        p_dev = torch.empty((4,), dtype=torch.float32, device=self.device)
        flag = torch.empty((4,), dtype=torch.int32, device=self.device)
        ws = torch.empty((abi.moe_savb_workspace_size(max(n_text, 1), d, hid),), dtype=torch.uint8,
                         device=self.device)
        exit_layer, trace = None, []
        for l in range(self.L):
            if exit_layer is None and l in gates and n_visual > 0 and n_text > 0:
                g = gates[l]
                abi.moe_savb_gate(src[n_visual:], g["w1"], g["b1"], g["w2"], g["b2"], theta, p_dev[:1],
                                  flag[:1], ws, stream=stream)
                fired = int(flag[0].item())  # host wait: the next layers' row count
                trace.append((l, float(p_dev[0].item())))
                if fired:
                    ht = self.hidden(n_text, "text")
                    abi.drop_visual_block_if(src, 0, n_visual, flag[:1], ht, stream=stream)
                    src, h, exit_layer = ht, ht, l
            dst = h if src is x else src
            self.layer_forward(l, src, dst, exit_layer is not None, p, stream=stream)
            src = dst
        return src, exit_layer, trace

    def capture_prefill(self, x: torch.Tensor, n_visual: int, p: float, gates: dict, theta: float):
        """Algorithm 2's prefill with the SAVB gate as ONE HIP graph over the
        static input rows x (packed bf16 layers).

        The exit layer is decided on the device, so from the first candidate
        layer on both variants of every layer are captured, each call
        predicated on the device int ``exit_layer`` (L = no exit yet):
          candidate l   moe_savb_gate_if runs while exit_layer == L and, when
                        it fires, sets exit_layer = l and its own flag; then
                        drop_visual_block_if copies the text rows when that
                        flag is set
          layer l       the dense block over all rows while exit_layer > l,
                        the RCEP block over the text rows while exit_layer <= l
        Layers before the first candidate run dense without a predicate.
        Returns a PrefillGraph: replay() runs the step; result() (one host
        read, after the replay) gives what forward_gated returns.
        """
        if not self.layers or not all(lay.packed and lay.w_r_packed is not None for lay in self.layers):
            raise ValueError("the captured prefill needs packed bf16 layers")
        T = x.shape[0]
        n_text = T - n_visual
        L = self.L
        dev = self.device
        cands = sorted(l for l in gates if 0 <= l < L) if n_visual > 0 and n_text > 0 else []
        hid = next(iter(gates.values()))["w1"].shape[0] if gates else 1
        st = _PrefillState(self, x, n_visual, cands, hid, dev)
        side = torch.cuda.Stream(device=dev)
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):  # every buffer exists before capture
            self._record_prefill(st, p, gates, theta)
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            self._record_prefill(st, p, gates, theta)
        st.graph = g
        return st

    def _record_prefill(self, st: "_PrefillState", p: float, gates: dict, theta: float):
        L, nv = self.L, st.n_visual
        st.exit_layer.fill_(L)  # fill kernels, not memsets (the graph replays them)
        st.fire.zero_()
        st.p_exit.zero_()
        h_full, h_text = self.hidden(st.T), self.hidden(st.T - nv, "text")
        first = st.cands[0] if st.cands else L
        never = (st.exit_layer, L, L + 1)  # no exit yet
        for l in range(L):
            src_full = st.x if l == 0 else h_full
            if l in st.cands:
                c = st.cands.index(l)
                gt = gates[l]
                abi.moe_savb_gate_if(src_full[nv:], gt["w1"], gt["b1"], gt["w2"], gt["b2"], theta,
                                     st.p_exit[c:c + 1], st.fire[c:c + 1], st.gate_ws, never,
                                     exit_layer=st.exit_layer, layer=l)
                abi.drop_visual_block_if(src_full, 0, nv, st.fire[c:c + 1], h_text)
            if l < first:
                self.layer_forward(l, src_full, h_full, False, p)
            else:
                self.layer_forward(l, src_full, h_full, False, p, guard=(st.exit_layer, l + 1, L + 1))
                self.layer_forward(l, h_text, h_text, True, p, guard=(st.exit_layer, 0, l + 1))

    def chainable(self) -> bool:
        """Every layer has packed bf16 weights (moe_rcep_layer_chained)."""
        return all(l.one_call for l in self.layers)

    def forward_decode(self, x: torch.Tensor, p: float, stream=None) -> torch.Tensor:
        """RCEP in every layer over x [T, d] with the layers' combines
        chained (forward with exit_layer 0 on a stack of packed layers):
        layer l's combine with the residual runs inside layer l + 1's first
        launch (moe_rcep_layer_chained), the last layer's as
        moe_combine_residual.  Returns the final hidden rows (a buffer owned
        by the stack)."""
        if not self.chainable():
            raise ValueError("chained decode needs packed bf16 layers")
        return self.forward(x, 0, p, exit_layer=0, stream=stream)

    def capture_decode(self, x: torch.Tensor, p: float):
        """Capture one decode step (RCEP in every layer, forward with
        exit_layer 0: the chained layers where every layer is packed) over
        the static input rows x as a HIP graph.  Returns (graph, out): replaying the graph
        reads x and leaves the final hidden rows in out."""
        run = lambda: self.forward(x, 0, p, exit_layer=0)  # noqa: E731
        side = torch.cuda.Stream(device=self.device)
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            run()  # buffers exist before capture
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            out = run()
        return g, out


class _PrefillState:
    """Device state and outputs of a captured prefill (MoEStack.capture_prefill)."""

    def __init__(self, stack: MoEStack, x: torch.Tensor, n_visual: int, cands: list, hid: int, dev):
        self.stack, self.x, self.n_visual, self.cands = stack, x, n_visual, cands
        self.T = x.shape[0]
        # exit_layer, and one flag and p_exit per candidate (16-byte rows)
        self.exit_layer = torch.empty((4,), dtype=torch.int32, device=dev)[:1]
        nc = max(len(cands), 1)
        self._fire = torch.zeros((nc, 4), dtype=torch.int32, device=dev)
        self._p = torch.zeros((nc, 4), dtype=torch.float32, device=dev)
        self.fire = self._fire[:, 0]
        self.p_exit = self._p[:, 0]
        n_text = self.T - n_visual
        self.gate_ws = torch.empty((abi.moe_savb_workspace_size(max(n_text, 1), x.shape[1], hid),),
                                   dtype=torch.uint8, device=dev)
        self.graph = None

    def replay(self):
        self.graph.replay()

    def result(self):
        """(final rows, exit layer or None, [(candidate, p_exit)] evaluated),
        as MoEStack.forward_gated returns them (reads the device state)."""
        torch.cuda.current_stream().synchronize()
        ex = int(self.exit_layer.item())
        L = self.stack.L
        ps = self._p[:, 0].cpu().tolist()
        evaluated = [(l, ps[i]) for i, l in enumerate(self.cands) if ex == L or l <= ex]
        if ex < L:
            return self.stack.hidden(self.T - self.n_visual, "text"), ex, evaluated
        return self.stack.hidden(self.T), None, evaluated
