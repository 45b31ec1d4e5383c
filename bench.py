#!/usr/bin/env python3
"""MoE-layer throughput of the RCEP hot path on one MI355X.

One step is one prefill of the Qwen3-VL-MoE-shaped MoE layer through the
visual exit (Algorithm 2 of the paper), on synthetic inputs already
resident in HBM:

  dense span   moe_route -> moe_dispatch -> moe_expert_ffn -> moe_combine
               (bf16: moe_route_packed, moe_dispatch without the row copy,
               moe_expert_ffn_packed_gather reading the token rows itself)
               over 4096 rows (3584 visual + 512 text), all 128 experts
  SAVB exit    drop_visual_block removes the 3584 visual rows
  RCEP span    moe_rcep_layer over the 512 text rows: full-pool routing,
               s and K with p = 0.9, the prefix re-route and the grouping,
               the expert FFN over experts [0, K), the combine

value = MoE-layer tokens per second over the step (4096 + 512 rows per
step).  In the timed steps every call of the dense span is bracketed by HIP
events on the stream it runs on, giving its stage times and the roofline of
the dominant kernel (the expert FFN); the RCEP span's stages are timed in a
second pass that runs them as separate calls (moe_route_rcep,
moe_expert_ffn_packed_gather, moe_combine).  The CPU oracle is timed on the
same step as the CPU baseline.

Other workloads (one JSON line each, same fields):

  --workload stack48   48-layer stack over 7680 visual + 512 text rows, exit
                       at layer 20 (dense layers 0-19 on 8192 rows, RCEP
                       layers 20-47 on 512 rows, p = 0.9); value = prefill
                       tokens/s through the 48 MoE layers
  --workload decode64  64 decode tokens through the same 48 layers, RCEP in
                       every layer (p = 0.85), one HIP graph per step;
                       value = decode tokens/s
  --workload stress    routing, dispatch and combine of the same layer at
                       65536 rows (bandwidth shape); value = rows/s
  --workload variants  synthetic analogs of the component ablation (dense,
                       visual exit only, fixed exit at 28, fixed prefix of
                       50, full) on the 48-layer stack, expert orders at
                       keep ratios and the p sweep; value = speedup of the
                       full method over the dense stack
  --workload gemm_ceiling
                       the expert FFN with every row on one expert (weights
                       cache-resident) at 32768 and 65536 rows, beside the
                       same SwiGLU through torch.matmul (the vendor GEMM
                       library) on the same shapes; value = the packed FFN's
                       TFLOP/s at 32768 rows

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline]
                       [--workload layer|stack48|decode64|stress|variants|gemm_ceiling]
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "MoE-layer tokens/s + % bf16 MFMA peak, dense 128-expert vs RCEP-prefix span"
PEAK_BF16_TFLOPS = 2500.0  # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0  # MI355X HBM3E


def stage_flops_bytes(stage: str, T: int, d: int, E: int, m: int, k: int, touched: int, K: int,
                      gather: bool = True):
    """Algorithmic FLOPs and HBM bytes of one ABI call (bf16 rows, fp32
    router and routing arrays).  Sizes per row and per expert are listed in
    the design notes.  With `gather` (layers on packed weights) the dispatch
    only groups the assignments and the expert GEMM reads the token rows
    through src_of_row; otherwise the dispatch copies them to x_perm."""
    A = T * k
    if stage == "route_full":
        return 2.0 * T * d * E, T * d * 2 + d * E * 4 + E * 4 + T * E * 4 + 2 * T * k * 4
    if stage == "route_prefix":
        return 0.0, T * K * 4 + 2 * T * k * 4
    if stage == "calibrate":
        return 0.0, 2 * T * k * 4 + E * 8 + 4
    if stage == "calibrate_route":  # masses, K and the prefix re-route in one call
        return 0.0, 2 * T * k * 4 + E * 8 + 4 + T * K * 4 + 2 * T * k * 4
    if stage == "route_rcep":  # router + full-pool Top-k + masses, K, re-route + grouping in one call
        f, b = stage_flops_bytes("route_full", T, d, E, m, k, touched, K, gather)
        _, b2 = stage_flops_bytes("calibrate_route", T, d, E, m, k, touched, K, gather)
        _, b3 = stage_flops_bytes("dispatch", T, d, E, m, k, touched, K, gather)
        return f, b + b2 + b3
    if stage == "dispatch":
        return 0.0, T * k * 4 + (E + 1) * 8 + 2 * A * 4 + (0 if gather else T * d * 2 + A * d * 2)
    if stage == "ffn":
        rows_in = T * d * 2 + A * 4 if gather else A * d * 2
        return 6.0 * A * d * m, touched * 3 * d * m * 2 + rows_in + A * d * 2 + (E + 1) * 4
    if stage == "combine":
        return 2.0 * A * d, A * d * 2 + A * 4 + A * 4 + T * d * 2
    if stage == "drop":
        return 0.0, 2 * T * d * 2  # T = rows kept
    raise KeyError(stage)


def roofline(flops: float, nbytes: float, sec: float) -> dict:
    t_mfma = flops / (PEAK_BF16_TFLOPS * 1e12)
    t_hbm = nbytes / (PEAK_HBM_GBS * 1e9)
    if flops > 0 and t_mfma >= t_hbm:
        ach = flops / sec / 1e12
        return dict(bound="mfma", achieved=ach, peak=PEAK_BF16_TFLOPS, unit="TFLOP/s",
                    frac=ach / PEAK_BF16_TFLOPS)
    ach = nbytes / sec / 1e9
    return dict(bound="hbm", achieved=ach, peak=PEAK_HBM_GBS, unit="GB/s", frac=ach / PEAK_HBM_GBS)


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_moe_expert_ffn_qwen3vl_4096.json")


def _counter_record():
    """The committed counter passes' summary, or None when the GEMM sources
    changed since they were taken."""
    try:
        from paper_2609_38823_amd.profiling import source_hash
        rec = json.load(open(TRAFFIC_FILE))
        return rec if rec.get("source_sha256") == source_hash() else None
    except (OSError, ValueError):
        return None


def measured_traffic():
    """HBM bytes per FFN call from the committed counter passes, or None."""
    rec = _counter_record()
    return rec.get("traffic_bytes_per_call") if rec else None


def measured_counters():
    """MFMA counters of the expert GEMM and per-stage achieved GB/s of the
    dense span at 4096 rows from the committed counter passes, or None."""
    rec = _counter_record()
    if not rec:
        return None
    m = rec.get("mfma") or {}
    return dict(
        mfma_busy_frac_at_peak_clock=m.get("mfma_busy_frac_at_peak_clock"),
        mfma_util_rocprof=m.get("mfma_util_rocprof"),
        mfma_flops_executed=m.get("mfma_flops_executed"),
        stages_hbm_frac={r["stage"]: round(r["hbm_frac"], 3) for r in rec.get("stages", [])},
        source="profiles/traffic_moe_expert_ffn_qwen3vl_4096.txt (rocprofv3 --pmc passes)")


def cpu_info() -> dict:
    info = {"affinity_cores": len(os.sched_getaffinity(0))}
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                info["model"] = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    try:
        from threadpoolctl import threadpool_info
        blas = [p for p in threadpool_info() if p.get("user_api") == "blas"]
        if blas:
            info["blas"] = blas[0].get("internal_api")
            info["blas_threads"] = blas[0].get("num_threads")
    except Exception:
        pass
    return info


def run_oracle_step(x, text, params, k, p):
    """The same step on the CPU oracle (test infrastructure, timed only):
    its step functions called in the order of the layer, each timed.
    Returns (total seconds, seconds per stage)."""
    import oracle
    import numpy as _np
    wr, b, gu, dn = params["w_r"], params["bias"], params["w_gate_up"], params["w_down"]
    E = wr.shape[1]
    st = {}

    def timed(name, fn, *a):
        t = time.perf_counter()
        r = fn(*a)
        st[name] = st.get(name, 0.0) + time.perf_counter() - t
        return r

    def experts(xr, idx, w, K=None):
        counts, offsets, src, ros = timed("dispatch", oracle.dispatch, idx, E)
        exp_of_row = _np.asarray(idx).reshape(-1)[src]
        y = timed("expert_ffn", oracle.expert_ffn_rows, _np.asarray(xr, _np.float64)[src // k], exp_of_row,
                  gu, dn)
        return timed("combine", oracle.combine, y, ros, w)

    t0 = time.perf_counter()
    a = timed("router_logits", oracle.router_logits, x, wr, b)
    idx, w = timed("topk", oracle.full_pool_route, a, k)
    experts(x, idx, w)
    h = timed("drop", oracle.drop_visual_block, x, 0, x.shape[0] - text.shape[0])
    a = timed("router_logits", oracle.router_logits, h, wr, b)
    idx_f, w_f = timed("topk", oracle.full_pool_route, a, k)
    mass = timed("mass_and_K", oracle.activated_mass, idx_f, w_f, E)
    K = timed("mass_and_K", oracle.prefix_length, mass, p, k)
    idx, w = timed("prefix_reroute", oracle.prefix_route, a, K, k)
    experts(h, idx, w)
    return time.perf_counter() - t0, {n: round(v, 4) for n, v in st.items()}


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--traffic-run", action="store_true",
                    help="only run the dense layer and a known-size copy (for rocprofv3 counter passes)")
    ap.add_argument("--workload", default="layer",
                    choices=["layer", "stack48", "decode64", "stress", "variants", "gemm_ceiling"])
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: the path has no multi-GPU execution "
              "(the design notes describe how it would shard); run with --gpus 1", file=sys.stderr)
        return 2
    fn = {"layer": bench_layer, "stack48": bench_stack48, "decode64": bench_decode64,
          "stress": bench_stress, "variants": bench_variants,
          "gemm_ceiling": bench_gemm_ceiling}[args.workload]
    return fn(args)


def bench_layer(args) -> int:
    import torch

    from paper_2609_38823_amd import abi, inputs as I
    from paper_2609_38823_amd.layer import MoELayer, apply_order, calibrate_order_router

    if not os.path.exists(abi.LIB_PATH):
        from paper_2609_38823_amd import build
        build.build()
    abi.load()
    torch.cuda.set_device(0)

    wl_d, wl_r = I.WORKLOADS["qwen3vl_dense_4096"], I.WORKLOADS["qwen3vl_rcep_512"]
    sh = wl_d.shape
    T, V, p = wl_d.T, wl_d.n_visual, wl_r.p
    d, E, m, k = sh.d, sh.E, sh.m, sh.k
    t_setup = time.perf_counter()
    prm = I.layer_params(sh, seed=wl_d.seed)
    x_np = I.tokens(sh, T, seed=wl_d.seed)
    x = torch.from_numpy(x_np).cuda().to(torch.bfloat16)
    # offline calibration on the 512 text rows, then the physical reorder
    order = calibrate_order_router(x[V:].contiguous(), prm["w_r"], prm["bias"], k)
    rprm = apply_order(prm, order)
    layer = MoELayer(rprm, k, sh.dtype)
    bd = layer.buffers(T)
    br = layer.buffers(T - V)
    h_text = torch.empty((T - V, d), dtype=torch.bfloat16, device="cuda")
    setup_s = time.perf_counter() - t_setup

    if args.traffic_run:
        # the FFN as the bench calls it, then a plain copy of a known size
        # (drop_visual_block with no rows dropped) for the counter scale
        for _ in range(3):
            layer.forward_dense(x, bd)
        src = torch.empty((65536, 2048), dtype=torch.bfloat16, device="cuda").fill_(1.0)
        dst = torch.empty_like(src)
        flush = torch.empty((1 << 30,), dtype=torch.uint8, device="cuda").fill_(0)  # evict src from caches
        del flush
        abi.drop_visual_block(src, 0, 0, dst)
        torch.cuda.synchronize()
        return 0

    stream = torch.cuda.current_stream()
    stages = ["route_full", "dispatch", "ffn", "combine", "drop", "r.route_rcep", "r.ffn", "r.combine"]

    def step(ev=None, rcep_stages=False):
        """One step.  With `ev` (len(stages) + 1 events): an event at the
        start, after each stage of the dense span and the drop, and at the
        end; with rcep_stages also between the RCEP span's stages, which then
        run as separate calls (routing, FFN, combine) instead of the one-call
        layer."""
        marks = iter(ev) if ev is not None else None

        def mark():
            if marks is not None:
                next(marks).record(stream)

        mark()
        layer.forward_dense(x, bd, mark=mark)
        abi.drop_visual_block(x, 0, V, h_text)
        mark()
        layer.forward_rcep(h_text, p, b=br, mark=mark if rcep_stages else None)
        if ev is not None and not rcep_stages:
            ev[-1].record(stream)

    def events(n):
        return [[torch.cuda.Event(enable_timing=True) for _ in range(len(stages) + 1)] for _ in range(n)]

    def mean_ms(evl, i, j):
        return float(np.mean([e[i].elapsed_time(e[j]) for e in evl]))

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    evs = events(args.steps)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(args.steps):
        step(evs[s])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = wall * 1e3 / args.steps
    # the RCEP span's stages: the same steps again with events between them
    evp = events(args.steps)
    for s in range(args.steps):
        step(evp[s], rcep_stages=True)
    torch.cuda.synchronize()
    n_dense = stages.index("r.route_rcep")
    stage_ms = {name: mean_ms(evs if i < n_dense else evp, i, i + 1) for i, name in enumerate(stages)}
    rcep_span_ms = mean_ms(evs, n_dense, len(stages))

    # the same step with the caches flushed first: a 512 MiB fill (twice the
    # memory-side cache) before each step, each step timed by its own events
    flush = torch.empty((512 << 20,), dtype=torch.uint8, device="cuda")
    n_cold = min(args.steps, 10)
    evc, evcp = events(n_cold), events(n_cold)
    for s in range(n_cold):
        flush.fill_(s & 0xFF)
        step(evc[s])
    for s in range(n_cold):
        flush.fill_(s & 0xFF)
        step(evcp[s], rcep_stages=True)
    torch.cuda.synchronize()
    del flush
    warm_span = mean_ms(evs, 0, len(stages))
    cold_span = mean_ms(evc, 0, len(stages))
    cold_stage = {name: round(mean_ms(evc if i < n_dense else evcp, i, i + 1), 4) for i, name in enumerate(stages)}
    cache = {"warm_event_ms_per_step": round(warm_span, 4), "cold_event_ms_per_step": round(cold_span, 4),
             "cold_tokens_per_s": (T + (T - V)) / (cold_span * 1e-3),
             "cold_stage_ms": cold_stage, "cold_steps": n_cold,
             "flush": "a 512 MiB fill before each cold step (the memory-side cache holds 256 MiB)"}

    # dense span over the 512 text rows alone (RCEP off), for the comparison
    K = int(br.K.cpu()[0])
    touched_d = int((bd.counts.cpu() > 0).sum())
    touched_r = int((br.counts.cpu() > 0).sum())
    from paper_2609_38823_amd.layer import Buffers
    bx = Buffers(T - V, d, E, m, k, torch.bfloat16)
    for _ in range(args.warmup):
        layer.forward_dense(h_text, bx)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(args.steps):
        layer.forward_dense(h_text, bx)
    e1.record(stream)
    torch.cuda.synchronize()
    dense512_ms = e0.elapsed_time(e1) / args.steps

    touched_512 = int((bx.counts.cpu() > 0).sum())

    # the paper's dense-equivalent executor on the RCEP span (App. A.3): every
    # text token through all K retained experts, weights applied afterwards
    from paper_2609_38823_amd.layer import Buffers as _B
    Tt = T - V
    bq = _B(Tt, d, E, m, E, torch.bfloat16, x_perm=False)
    idx_d = torch.empty((Tt, E), dtype=torch.int32, device="cuda")
    w_d = torch.empty((Tt, E), dtype=torch.float32, device="cuda")

    def dense_equiv():
        abi.moe_expand_dense_routing(br.idx, br.w, E, idx_d, w_d, K_dev=br.K)
        abi.moe_dispatch(idx_d, E, None, bq.counts, bq.offsets, bq.src_of_row, bq.row_of_slot,
                         None, bq.ws)
        abi.moe_expert_ffn_packed_gather(h_text, E, bq.src_of_row, bq.offsets, layer.w_gate_up,
                                         layer.w_down, bq.y_perm, bq.ws, K_dev=br.K)
        abi.moe_combine(bq.y_perm, bq.row_of_slot, w_d, bq.out)

    for _ in range(args.warmup):
        dense_equiv()
    e0.record(stream)
    for _ in range(args.steps):
        dense_equiv()
    e1.record(stream)
    torch.cuda.synchronize()
    dense_equiv_ms = e0.elapsed_time(e1) / args.steps

    def fb(stage, T_, touched, K_=E):
        return stage_flops_bytes(stage, T_, d, E, m, k, touched, K_)

    stage_rep = {}
    for name in stages:
        base = name.split(".")[-1]
        Tn = T if not name.startswith("r.") and base != "drop" else T - V
        f, b = fb(base, Tn, touched_r if name.startswith("r.") else touched_d, K)
        sec = stage_ms[name] * 1e-3
        stage_rep[name] = dict(ms=round(stage_ms[name], 4), roofline=roofline(f, b, sec),
                               gflop=round(f / 1e9, 3), mb=round(b / 1e6, 3))

    per_tok_flops = 2 * d * E + 6 * k * d * m
    dense_ms = sum(stage_ms[s] for s in ["route_full", "dispatch", "ffn", "combine"])
    rcep_ms = rcep_span_ms  # the one-call layer, as the timed step runs it
    spans = {
        "dense@4096": dict(ms=round(dense_ms, 4), tokens_per_s=T / dense_ms * 1e3,
                           tflops=per_tok_flops * T / dense_ms / 1e9, touched_experts=touched_d),
        "rcep@512": dict(ms=round(rcep_ms, 4), tokens_per_s=(T - V) / rcep_ms * 1e3,
                         tflops=per_tok_flops * (T - V) / rcep_ms / 1e9, K=K, touched_experts=touched_r,
                         paper_dense_equiv_tflops=(2 * d * E + 6 * K * d * m) * (T - V) / rcep_ms / 1e9,
                         separate_calls_ms=round(sum(stage_ms[s] for s in stages if s.startswith("r.")), 4)),
        "rcep@512 experts, dense-equivalent executor": dict(
            ms=round(dense_equiv_ms, 4), K=K, expert_gflop=6 * K * d * m * (T - V) / 1e9,
            sparse_expert_ms=round(stage_ms["r.ffn"] + stage_ms["r.combine"], 4),
            note="expand + dispatch (k = E) + expert FFN over experts [0, K) + combine; the RCEP "
                 "span's sparse FFN/combine for comparison (its grouping runs inside r.route_rcep)"),
        "dense@512": dict(ms=round(dense512_ms, 4), tokens_per_s=(T - V) / dense512_ms * 1e3,
                          tflops=per_tok_flops * (T - V) / dense512_ms / 1e9, touched_experts=touched_512,
                          paper_dense_equiv_tflops=(2 * d * E + 6 * E * d * m) * (T - V) / dense512_ms / 1e9),
    }
    f, b = fb("ffn", T, touched_d)
    ffn_roof = roofline(f, b, stage_ms["ffn"] * 1e-3)
    ffn_roof["traffic"] = measured_traffic()
    ffn_roof["counters"] = measured_counters()
    ffn_roof["kernel"] = ("moe_expert_ffn_packed_gather @ dense 4096 rows (gate/up GEMM reading the token "
                          "rows through src_of_row + down GEMM, on packed bf16 weights)")
    ffn_roof["mfma_frac"] = f / (stage_ms["ffn"] * 1e-3) / 1e12 / PEAK_BF16_TFLOPS

    cpu = None
    if not args.no_cpu_baseline:
        sec, stage_s = run_oracle_step(x_np, x_np[V:], rprm, k, p)
        info = cpu_info()
        cpu = dict(value=(T + (T - V)) / sec, unit="tokens/s",
                   cores=info.get("blas_threads") or info["affinity_cores"], kind="oracle",
                   sample="one full step (dense 4096 rows + visual drop + RCEP 512 rows), numpy float64",
                   seconds=round(sec, 3), stage_seconds=stage_s, **info)

    tokens = T + (T - V)
    line = {
        "metric": METRIC,
        "value": tokens / (ms_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "Qwen3-VL-MoE MoE layer (d 2048, 128 experts x 768, top-8, bf16, fp32 router): "
                               "dense span over 4096 rows (3584 visual + 512 text), SAVB drop of the visual "
                               "block, RCEP span over the 512 text rows (p 0.9)",
                   "tokens_per_step": tokens, "seed": wl_d.seed, "zipf_alpha": sh.zipf_alpha},
        "roofline": ffn_roof,
        "cpu_baseline": cpu,
        "spans": spans,
        "stages": stage_rep,
        "cache": cache,
        "setup_s": round(setup_s, 1),
    }
    print(json.dumps(line), flush=True)
    return 0


# --------------------------------------------------------------------------
# Other workloads
# --------------------------------------------------------------------------
def _setup_gpu():
    import torch

    from paper_2609_38823_amd import abi

    if not os.path.exists(abi.LIB_PATH):
        from paper_2609_38823_amd import build
        build.build()
    abi.load()
    torch.cuda.set_device(0)


def _log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def _build_stack(wl):
    from paper_2609_38823_amd.stack import MoEStack
    t0 = time.perf_counter()
    st = MoEStack(wl, progress=lambda l: _log(f"layer {l} loaded") if l % 8 == 7 else None)
    return st, time.perf_counter() - t0


def _line(metric, value, unit, args, ms_step, config, roof, cpu, **extra):
    line = {"metric": metric, "value": value, "unit": unit, "n_gpus": 1, "steps": args.steps,
            "warmup": args.warmup, "ms_per_step": ms_step, "higher_is_better": True,
            "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
            "config": config, "roofline": roof, "cpu_baseline": cpu}
    line.update(extra)
    print(json.dumps(line), flush=True)
    return 0


def _timed_layer(st, l, h, rcep, p, stream, reps=6):
    """One layer with events after each ABI call, run `reps` times back to
    back; returns the per-call median ms over the repetitions after the
    first (the GPU is then busy when each repetition's first event is
    recorded, so no host launch gap enters the times) and the buffers (h
    is left unmodified: the layer writes a scratch copy)."""
    import torch
    dst = torch.empty_like(h)
    runs = []
    b = None
    for _ in range(reps):
        used = [torch.cuda.Event(enable_timing=True)]
        used[0].record(stream)

        def mark():
            e = torch.cuda.Event(enable_timing=True)
            e.record(stream)
            used.append(e)

        b = st.layer_forward(l, h, dst, rcep, p, mark=mark)
        runs.append(used)
    torch.cuda.synchronize()
    per = [[u[i].elapsed_time(u[i + 1]) for i in range(len(u) - 1)] for u in runs[1:]]
    return [float(np.median(c)) for c in zip(*per)], b


def bench_stack48(args) -> int:
    """48-layer prefill: 20 dense layers over 8192 rows, the visual drop,
    28 RCEP layers over the 512 text rows."""
    import torch

    from paper_2609_38823_amd import inputs as I
    _setup_gpu()
    wl = I.WORKLOADS["qwen3vl_stack48_8192"]
    sh = wl.shape
    d, E, m, k = sh.d, sh.E, sh.m, sh.k
    st, setup_s = _build_stack(wl)
    x_np = I.tokens(sh, wl.T, seed=wl.seed)
    x = torch.from_numpy(x_np).cuda().to(torch.bfloat16)
    stream = torch.cuda.current_stream()
    for _ in range(args.warmup):
        st.forward(x, wl.n_visual, wl.p, wl.exit_layer)
    torch.cuda.synchronize()
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    evs[0].record(stream)
    for s in range(args.steps):
        st.forward(x, wl.n_visual, wl.p, wl.exit_layer)
        evs[s + 1].record(stream)
    torch.cuda.synchronize()
    step_ms = [evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps)]
    ms = float(np.mean(step_ms))
    Ks = st.K_trace[:, 0].cpu().numpy()[wl.exit_layer:]
    # per-call times of one dense layer (8192 rows) and one RCEP layer (512)
    h_text = torch.empty((wl.T - wl.n_visual, d), dtype=torch.bfloat16, device="cuda")
    from paper_2609_38823_amd import abi
    abi.drop_visual_block(x, 0, wl.n_visual, h_text)
    dense_calls, bd = _timed_layer(st, 0, x, False, wl.p, stream)
    rcep_calls, br = _timed_layer(st, wl.exit_layer, h_text, True, wl.p, stream)
    touched = int((bd.counts.cpu() > 0).sum())
    K20 = int(st.K_trace[wl.exit_layer, 0].cpu())
    # one SAVB gate evaluation (Eqs. 2-3) on the 512 text rows entering a
    # candidate layer: the cost a gate-decided exit adds per candidate
    gp = I.gate_params(d, seed=wl.seed, layer=wl.exit_layer)
    gd = {k2: torch.from_numpy(v).cuda() for k2, v in gp.items()}
    text_rows = x[wl.n_visual:]
    g_p = torch.empty((4,), dtype=torch.float32, device="cuda")
    g_f = torch.empty((4,), dtype=torch.int32, device="cuda")
    g_ws = torch.empty((abi.moe_savb_workspace_size(wl.T - wl.n_visual, d, 512),), dtype=torch.uint8,
                       device="cuda")
    for _ in range(3):
        abi.moe_savb_gate(text_rows, gd["w1"], gd["b1"], gd["w2"], gd["b2"], 0.5, g_p[:1], g_f[:1], g_ws)
    # one call at a time on an idle stream (as in the stack, where the flag is
    # read after each evaluation): event time from the call's start to the
    # end of its four launches, launch latency included
    g_t = []
    for _ in range(20):
        g0, g1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        g0.record(stream)
        abi.moe_savb_gate(text_rows, gd["w1"], gd["b1"], gd["w2"], gd["b2"], 0.5, g_p[:1], g_f[:1], g_ws)
        g1.record(stream)
        torch.cuda.synchronize()
        g_t.append(g0.elapsed_time(g1))
    gate_us = float(np.median(g_t)) * 1e3
    graph = _captured_prefill(st, x, wl, d, stream, max(3, args.steps // 2))
    f, b = stage_flops_bytes("ffn", wl.T, d, E, m, k, touched, E)
    ffn_ms = dense_calls[2]
    roof = roofline(f, b, ffn_ms * 1e-3)
    roof["kernel"] = "moe_expert_ffn_packed_gather @ dense 8192 rows (layer 0 of the stack)"
    roof["traffic"] = None
    roof["mfma_frac"] = f / (ffn_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS
    per_tok = 2 * d * E + 6 * k * d * m
    alg_flops = per_tok * (wl.T * wl.exit_layer + (wl.T - wl.n_visual) * (wl.layers - wl.exit_layer))
    cpu = None
    if not args.no_cpu_baseline:
        cpu = _oracle_stack_sample(st, x_np, wl)
    names_d = ["route", "dispatch", "ffn", "combine_residual"]
    names_r = ["route_rcep", "ffn", "combine_residual"]
    return _line(
        "MoE-stack prefill tokens/s (48 MoE layers, SAVB exit at layer 20, RCEP p 0.9)",
        wl.T / (ms * 1e-3), "tokens/s", args, ms,
        {"workload": "Qwen3-VL-MoE 48-layer MoE stack (d 2048, 128 experts x 768, top-8, bf16): "
                     "8192 prefill rows (7680 visual + 512 text); layers 0-19 dense over 8192 rows, "
                     "visual rows dropped at the entrance of layer 20, layers 20-47 RCEP over 512 rows",
         "seed": wl.seed, "zipf_alpha": sh.zipf_alpha, "exit_layer": wl.exit_layer},
        roof, cpu,
        tflops=alg_flops / (ms * 1e-3) / 1e12, K_per_rcep_layer=[int(v) for v in Ks],
        K_mean=float(np.mean(Ks)), step_ms_min=float(np.min(step_ms)),
        dense_layer_8192={n: round(v, 4) for n, v in zip(names_d, dense_calls)},
        rcep_layer_512={n: round(v, 4) for n, v in zip(names_r, rcep_calls)},
        paper_flops_replay=paper_prefill_flops(wl.T, wl.T - wl.n_visual, wl.exit_layer, Ks, wl.layers, E, d, m,
                                               n_gate=len(range(0, wl.exit_layer, 4)) + 1),
        touched_dense=touched, K_rcep_layer_512=K20, savb_gate_us=round(gate_us, 2),
        savb_gate_candidates_before_exit=len(range(0, wl.exit_layer, 4)), captured_prefill=graph,
        setup_s=round(setup_s, 1))


def _captured_prefill(st, x, wl, d, stream, reps):
    """Algorithm 2's prefill with the SAVB gate as one captured HIP graph
    (MoEStack.capture_prefill): gates before every fourth layer, biased so
    that the one before the workload's exit layer fires, timed beside the
    eager gated prefill (which reads each candidate's flag on the host)."""
    import torch

    from paper_2609_38823_amd import inputs as I
    gates = {}
    for l in range(0, wl.layers, 4):
        g = {k2: torch.from_numpy(v).cuda() for k2, v in I.gate_params(d, seed=wl.seed, layer=l).items()}
        hi = 20.0 if l == wl.exit_layer else -20.0
        g["b2"].copy_(torch.tensor([-hi, hi], dtype=torch.float32))
        gates[l] = g

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            fn()
            e1.record(stream)
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1))
        return float(np.median(ts))

    eager_ms = timed(lambda: st.forward_gated(x, wl.n_visual, wl.p, gates, 0.5))
    out_e, ex_e, _ = st.forward_gated(x, wl.n_visual, wl.p, gates, 0.5)
    ref = out_e.clone()
    pg = st.capture_prefill(x, wl.n_visual, wl.p, gates, 0.5)
    graph_ms = timed(pg.replay)
    out_g, ex_g, _ = pg.result()
    same = ex_g == ex_e and torch.equal(out_g.view(torch.int16), ref.view(torch.int16))
    return dict(graph_ms=round(graph_ms, 3), eager_gated_ms=round(eager_ms, 3), exit_layer=ex_g,
                candidates=len(gates), bitwise_equal_to_eager=bool(same),
                tokens_per_s=round(wl.T / (graph_ms * 1e-3), 1))


def paper_prefill_flops(S: int, T: int, exit_layer: int, Ks, L: int, E: int, d: int, m: int,
                        n_gate: int = 0) -> dict:
    """The paper's decoder FLOPs replay for one prefill (App. A.3), from
    paper_2609_38823_amd.flops: layers before the exit at (S, E), from the
    exit on at (T, K_l); the baseline runs every layer at (S, E)."""
    from paper_2609_38823_amd import flops as F
    g = F.DecoderDims(d=d, E=E, m=m)
    c = F.case_flops(g, L=L, S=S, V=S - T, exit_layer=exit_layer, K_prefill=[int(K) for K in Ks],
                     n_gate=n_gate)
    return dict(baseline_tflop=c["baseline"] / 1e12, decomoe_tflop=c["method"] / 1e12,
                gate_tflop=c["method_gate"] / 1e12, saving=F.saving([c]), q=g.q, kv=g.kv,
                convention="paper's replay: dense-equivalent experts (6 K d m per token), attention "
                           "terms included, one prefill, exit at the given layer")


def _oracle_stack_sample(st, x_np, wl):
    """The oracle on one dense layer (8192 rows) and one RCEP layer (512
    rows) of the stack, extrapolated to the stack's 20 + 28 layers."""
    import oracle
    import torch

    from paper_2609_38823_amd import inputs as I

    def params(l):
        rp = I.router_params(st.sh, wl.seed, l)
        gu, dn = I.device_expert_weights(st.sh, wl.seed, l)
        gu_h, dn_h = gu.float().cpu().numpy(), dn.float().cpu().numpy()
        del gu, dn
        torch.cuda.empty_cache()
        w_r, bias, wgu, wd = oracle.permute_experts(st.orders[l], rp["w_r"], rp["bias"], gu_h, dn_h)
        return w_r, bias, wgu, wd

    k = st.sh.k
    w_r, bias, wgu, wd = params(0)
    t0 = time.perf_counter()
    oracle.moe_layer_dense(x_np, w_r, bias, wgu, wd, k)
    t_dense = time.perf_counter() - t0
    w_r, bias, wgu, wd = params(wl.exit_layer)
    t0 = time.perf_counter()
    oracle.moe_layer_rcep(x_np[wl.n_visual:], w_r, bias, wgu, wd, k, wl.p)
    t_rcep = time.perf_counter() - t0
    sec = t_dense * wl.exit_layer + t_rcep * (wl.layers - wl.exit_layer)
    info = cpu_info()
    return dict(value=wl.T / sec, unit="tokens/s", cores=info.get("blas_threads") or info["affinity_cores"],
                kind="oracle", sample=("one dense layer over 8192 rows and one RCEP layer over 512 rows, "
                                       "timed, extrapolated x20 + x28 (numpy float64)"),
                seconds_measured=round(t_dense + t_rcep, 3), extrapolated=True, **info)


def bench_decode64(args) -> int:
    """64 decode tokens through 48 RCEP layers, one HIP graph per step."""
    import torch

    from paper_2609_38823_amd import inputs as I
    _setup_gpu()
    wl = I.WORKLOADS["qwen3vl_decode64"]
    sh = wl.shape
    d, E, m, k = sh.d, sh.E, sh.m, sh.k
    st, setup_s = _build_stack(I.WORKLOADS["qwen3vl_stack48_8192"])
    x_np = I.tokens(sh, wl.T, seed=wl.seed, stream="decode")
    x = torch.from_numpy(x_np).cuda().to(torch.bfloat16)
    stream = torch.cuda.current_stream()
    # touched experts per layer (eager, outside the timed region)
    touched = []
    h = x.clone()
    for l in range(st.L):
        dst = torch.empty_like(h)
        b = st.layer_forward(l, h, dst, True, wl.p)
        touched.append(int((b.counts.cpu() > 0).sum()))
        h = dst
    Ks = st.K_trace[:, 0].cpu().numpy()
    # eager step time
    for _ in range(2):
        st.forward(x, 0, wl.p, exit_layer=0)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(args.steps):
        st.forward(x, 0, wl.p, exit_layer=0)
    e1.record(stream)
    torch.cuda.synchronize()
    eager_ms = e0.elapsed_time(e1) / args.steps
    g, _ = st.capture_decode(x, wl.p)
    for _ in range(args.warmup):
        g.replay()
    torch.cuda.synchronize()
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    evs[0].record(stream)
    for s in range(args.steps):
        g.replay()
        evs[s + 1].record(stream)
    torch.cuda.synchronize()
    step_ms = [evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps)]
    ms = float(np.mean(step_ms))
    A = wl.T * k
    wbytes = sum(t * 3 * d * m * 2 for t in touched)
    nbytes = wbytes + st.L * (2 * A * d * 2 + 3 * wl.T * d * 2 + d * E * 4)
    ach = nbytes / (ms * 1e-3) / 1e9
    roof = dict(bound="hbm", achieved=ach, peak=PEAK_HBM_GBS, unit="GB/s", frac=ach / PEAK_HBM_GBS,
                traffic=None, kernel="whole decode step (48 layers, weight streaming of touched experts)")
    variants = _decode_variants(st, x, wl, args, stream)
    cpu = None
    if not args.no_cpu_baseline:
        cpu = _oracle_decode_sample(st, x_np, wl)
    return _line(
        "MoE-stack decode tokens/s (64 tokens x 48 MoE layers, RCEP p 0.85, HIP graph)",
        wl.T / (ms * 1e-3), "tokens/s", args, ms,
        {"workload": "Qwen3-VL-MoE 48-layer MoE stack (d 2048, 128 experts x 768, top-8, bf16): "
                     "decode of 64 single text tokens, RCEP in all 48 layers, one K per layer",
         "seed": wl.seed, "zipf_alpha": sh.zipf_alpha},
        roof, cpu, eager_ms_per_step=eager_ms, step_ms_min=float(np.min(step_ms)),
        K_per_layer=[int(v) for v in Ks], touched_per_layer=touched,
        weight_bytes_per_step=wbytes, variants=variants, setup_s=round(setup_s, 1))


def _decode_variants(st, x, wl, args, stream):
    """Readings of the decode workload beside the batch-shared K (eager
    steps, outside the timed value): one invocation per sequence (each of
    the 64 tokens its own segment, so its own K; the expert FFN runs the
    experts below the largest K) and RCEP only from layer 20 (layers 0-19
    on the full pool)."""
    import torch

    T, E = x.shape[0], st.sh.E
    seg = torch.arange(T + 1, dtype=torch.int32, device=x.device)
    bufs = {}

    def per_sequence(record=None):
        h = x
        for l, layer in enumerate(st.layers):
            if l not in bufs:
                bufs[l] = (layer.buffers(T, T), torch.empty_like(x))
            b, dst = bufs[l]
            layer.forward_rcep(h, wl.p, seg_offsets=seg, b=b, residual=h, out=dst)
            if record is not None:
                record(l, b)
            h = dst
        return h

    Ks, touched = [], []
    per_sequence(lambda l, b: (Ks.append(b.K[:T].cpu().numpy().copy()),
                               touched.append(int((b.counts.cpu() > 0).sum()))))
    Ks = np.stack(Ks)

    def timed(fn):
        for _ in range(2):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(args.steps):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / args.steps

    ms_seq = timed(per_sequence)
    ms_20 = timed(lambda: st.forward(x, 0, wl.p, exit_layer=20))
    K20 = st.K_trace[20:, 0].cpu().numpy()
    return {
        "per-sequence K (64 invocations of one token)": dict(
            ms_per_step=round(ms_seq, 3), tokens_per_s=T / (ms_seq * 1e-3),
            K_min=int(Ks.min()), K_median=float(np.median(Ks)), K_max=int(Ks.max()),
            touched_mean=float(np.mean(touched)), touched_per_layer=touched),
        "RCEP from layer 20 (layers 0-19 on all experts)": dict(
            ms_per_step=round(ms_20, 3), tokens_per_s=T / (ms_20 * 1e-3), K_mean_from_20=float(K20.mean())),
    }


def _oracle_decode_sample(st, x_np, wl):
    """The oracle's decode over the first 4 layers, extrapolated to 48."""
    import oracle
    import torch

    from paper_2609_38823_amd import inputs as I
    n = 4
    sec = 0.0
    h = np.asarray(x_np, np.float64)
    for l in range(n):
        rp = I.router_params(st.sh, st.wl.seed, l)
        gu, dn = I.device_expert_weights(st.sh, st.wl.seed, l)
        gu_h, dn_h = gu.float().cpu().numpy(), dn.float().cpu().numpy()
        del gu, dn
        torch.cuda.empty_cache()
        w_r, bias, wgu, wd = oracle.permute_experts(st.orders[l], rp["w_r"], rp["bias"], gu_h, dn_h)
        t0 = time.perf_counter()
        h = h + oracle.moe_layer_rcep(h, w_r, bias, wgu, wd, st.sh.k, wl.p)["out"]
        sec += time.perf_counter() - t0
    sec *= st.L / n
    info = cpu_info()
    return dict(value=wl.T / sec, unit="tokens/s", cores=info.get("blas_threads") or info["affinity_cores"],
                kind="oracle", sample="decode of the 64 tokens through layers 0-3, timed, extrapolated x12 "
                                      "(numpy float64)", extrapolated=True, **info)


def bench_stress(args) -> int:
    """Routing, dispatch and combine of the layer at 65536 rows."""
    import torch

    from paper_2609_38823_amd import abi, inputs as I
    from paper_2609_38823_amd.layer import Buffers, to_device
    _setup_gpu()
    wl = I.WORKLOADS["qwen3vl_dense_4096"]
    sh = wl.shape
    d, E, m, k = sh.d, sh.E, sh.m, sh.k
    T = 65536
    rp = I.router_params(sh, wl.seed)
    w_r, bias = to_device(rp["w_r"], torch.float32), to_device(rp["bias"], torch.float32)
    w_rp = torch.empty((3 * d * E,), dtype=torch.bfloat16, device="cuda")
    abi.moe_pack_router(w_r, w_rp)
    x = to_device(I.tokens(sh, T, seed=1), torch.bfloat16)
    b = Buffers(T, d, E, m, k, torch.bfloat16)
    stream = torch.cuda.current_stream()
    names = ["route_full", "dispatch", "combine"]

    def step(ev=None):
        it = iter(ev) if ev is not None else None

        def mark():
            if it is not None:
                next(it).record(stream)

        mark()
        abi.moe_route_packed(x, w_rp, bias, k, b.logits, b.idx, b.w, ws=b.ws)
        mark()
        abi.moe_dispatch(b.idx, E, x, b.counts, b.offsets, b.src_of_row, b.row_of_slot, b.x_perm, b.ws)
        mark()
        abi.moe_combine(b.x_perm, b.row_of_slot, b.w, b.out)  # dispatched rows stand in for y_perm
        mark()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    for s in range(args.steps):
        step(evs[s])
    torch.cuda.synchronize()
    st_ms = {n: float(np.mean([e[i].elapsed_time(e[i + 1]) for e in evs])) for i, n in enumerate(names)}
    ms = sum(st_ms.values())
    rep = {}
    for n in names:
        f, nb = stage_flops_bytes(n, T, d, E, m, k, E, E, gather=False)
        rep[n] = dict(ms=round(st_ms[n], 4), roofline=roofline(f, nb, st_ms[n] * 1e-3),
                      gflop=round(f / 1e9, 3), mb=round(nb / 1e6, 3))
    # the router runs the float32 product as three bf16 MFMA terms: its
    # binding floor is the larger of the stage's HBM bytes and that executed
    # MFMA work at peak
    f, nb = stage_flops_bytes("route_full", T, d, E, m, k, E, E, gather=False)
    sec = st_ms["route_full"] * 1e-3
    floor = max(nb / (PEAK_HBM_GBS * 1e9), 3 * f / (PEAK_BF16_TFLOPS * 1e12))
    rep["route_full"]["split_router"] = dict(
        executed_gflop=round(3 * f / 1e9, 3), executed_mfma_frac=round(3 * f / sec / 1e12 / PEAK_BF16_TFLOPS, 4),
        floor_us=round(floor * 1e6, 2), frac_of_floor=round(floor / sec, 4))
    f, nb = stage_flops_bytes("dispatch", T, d, E, m, k, E, E, gather=False)
    roof = roofline(f, nb, st_ms["dispatch"] * 1e-3)
    roof["kernel"] = "moe_dispatch @ 65536 rows (counting sort + row gather)"
    roof["traffic"] = None
    return _line(
        "Routing + dispatch + combine rows/s at 65536 rows (bandwidth shape of the MoE layer)",
        T / (ms * 1e-3), "rows/s", args, ms,
        {"workload": "Qwen3-VL-MoE MoE layer shape (d 2048, 128 experts, top-8, bf16, fp32 router) at "
                     "65536 rows: moe_route_packed (full pool), moe_dispatch, moe_combine (no expert FFN)",
         "seed": 1}, roof, None, stages=rep)


def bench_variants(args) -> int:
    """Component ablation analogs on the stack, expert-order analysis at
    keep ratios and the p sweep (one JSON line)."""
    import torch

    from paper_2609_38823_amd import abi, inputs as I
    from paper_2609_38823_amd.layer import MoELayer, apply_order, calibrate_order_router, to_device
    _setup_gpu()
    stream = torch.cuda.current_stream()
    wl = I.WORKLOADS["qwen3vl_stack48_8192"]
    sh = wl.shape
    d, E, m, k = sh.d, sh.E, sh.m, sh.k
    st, setup_s = _build_stack(wl)
    x_np = I.tokens(sh, wl.T, seed=wl.seed)
    x = torch.from_numpy(x_np).cuda().to(torch.bfloat16)
    Tt = wl.T - wl.n_visual

    def timed(fn):
        for _ in range(args.warmup):
            fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(args.steps):
            out = fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / args.steps, out

    variants = {
        "dense (no exit, all experts)": dict(exit_layer=None),
        "visual exit only (exit 20, all experts)": dict(exit_layer=20, after_exit="dense"),
        "fixed exit at 28 + RCEP": dict(exit_layer=28),
        "exit 20 + fixed prefix of 50": dict(exit_layer=20, after_exit="fixed", K_fixed=50),
        "exit 20 + RCEP (full)": dict(exit_layer=20),
    }
    rows = {}
    ref_text = None
    wbytes = 3 * d * m * 2
    for name, kw in variants.items():
        ms, out = timed(lambda: st.forward(x, wl.n_visual, wl.p, **kw))
        final = out.float()
        text = final[wl.n_visual:] if final.shape[0] == wl.T else final
        text = text.cpu().numpy().astype(np.float64)
        if ref_text is None:
            ref_text = text
        ex = kw.get("exit_layer")
        Ks = st.K_trace[:, 0].cpu().numpy()
        if ex is None:
            touched = [E] * st.L
        elif kw.get("after_exit") == "dense":
            touched = [E] * st.L
        elif kw.get("after_exit") == "fixed":
            touched = [E] * ex + [50] * (st.L - ex)
        else:
            touched = [E] * ex + [int(v) for v in Ks[ex:]]
        rows[name] = dict(ms=round(ms, 3), tokens_per_s=wl.T / ms * 1e3,
                          mean_experts_after_exit=float(np.mean(touched[ex:])) if ex is not None else float(E),
                          expert_weight_gb_per_step=sum(touched) * wbytes / 1e9,
                          text_rows_rel_l2_vs_dense=float(np.linalg.norm(text - ref_text) / np.linalg.norm(ref_text)))
    speedup = rows["dense (no exit, all experts)"]["ms"] / rows["exit 20 + RCEP (full)"]["ms"]

    # p sweep over the stack (exit 20): mean K of the 28 RCEP layers
    p_sweep = {}
    for pv in (0.1, 0.3, 0.5, 0.7, 0.8, 0.9, 0.95, 1.0):
        st.forward(x, wl.n_visual, pv, 20)
        Ks = st.K_trace[20:, 0].cpu().numpy()
        p_sweep[str(pv)] = dict(mean_K=float(Ks.mean()), min_K=int(Ks.min()), max_K=int(Ks.max()))

    # expert orders at keep ratios on one layer (the Qwen layer's 512 text
    # rows): routed mass covered by the first K experts of each order, and the
    # layer output with that fixed prefix against the full pool
    lw = I.WORKLOADS["qwen3vl_dense_4096"]
    prm = I.layer_params(sh, seed=lw.seed)
    xt_np = I.tokens(sh, lw.T, seed=lw.seed)[lw.n_visual:]
    xt = torch.from_numpy(xt_np).cuda().to(torch.bfloat16)
    orders = {"native": np.arange(E),
              "random": np.random.default_rng(7).permutation(E),
              "RCEP (Mean-Mass)": calibrate_order_router(xt, prm["w_r"], prm["bias"], k)}
    # activated mass per native expert from the full-pool routing (device)
    lay0 = MoELayer(prm, k, sh.dtype)
    b0 = lay0.forward_rcep(xt, 1.0)
    s_native = b0.mass[0].cpu().numpy()
    dense_out = lay0.forward_dense(xt).out.float().cpu().numpy().astype(np.float64)
    del lay0
    torch.cuda.empty_cache()
    keep = (0.1, 0.2, 0.3, 0.4, 0.5)
    order_rows = {}
    for oname, order in orders.items():
        lay = MoELayer(apply_order(prm, order), k, sh.dtype)
        s_o = s_native[order]
        res = {}
        for r in keep:
            K = int(round(r * E))
            out = lay.forward_prefix(xt, K).out.float().cpu().numpy().astype(np.float64)
            res[str(r)] = dict(K=K, mass_covered=float(s_o[:K].sum() / s_o.sum()),
                               weight_mb=K * wbytes / 1e6,
                               out_rel_l2_vs_full_pool=float(np.linalg.norm(out - dense_out) /
                                                             np.linalg.norm(dense_out)))
        order_rows[oname] = res
        del lay
        torch.cuda.empty_cache()

    return _line(
        "Synthetic component ablation: speedup of exit 20 + RCEP over the dense 48-layer stack",
        speedup, "x", args, rows["exit 20 + RCEP (full)"]["ms"],
        {"workload": "Qwen3-VL-MoE 48-layer MoE stack (d 2048, 128 experts x 768, top-8, bf16), 8192 "
                     "prefill rows (7680 visual + 512 text); order analysis on one layer's 512 text rows",
         "seed": wl.seed, "zipf_alpha": sh.zipf_alpha},
        None, None, ablation=rows, p_sweep_stack=p_sweep, orders_at_keep_ratio=order_rows,
        setup_s=round(setup_s, 1))



def bench_gemm_ceiling(args) -> int:
    """The packed expert FFN with all rows on one expert beside the vendor
    GEMM library (torch.matmul) on the same SwiGLU shapes: what a library
    bf16 GEMM reaches on this chip for the FFN's own contraction sizes."""
    import torch

    from paper_2609_38823_amd import abi, inputs as I
    from paper_2609_38823_amd.layer import MoELayer, to_device
    _setup_gpu()
    stream = torch.cuda.current_stream()
    wl = I.WORKLOADS["qwen3vl_dense_4096"]
    sh = wl.shape
    d, E, m, k = sh.d, sh.E, sh.m, sh.k
    prm = I.layer_params(sh, seed=wl.seed)
    layer = MoELayer(prm, k, sh.dtype)
    # expert 0's weights, row-major, for the library: right operands stored
    # contiguous as [K, N]
    wguT = to_device(prm["w_gate_up"][0], torch.bfloat16).t().contiguous()  # [d, 2m]
    wdnT = to_device(prm["w_down"][0], torch.bfloat16).t().contiguous()  # [m, d]

    def timed(fn):
        for _ in range(args.warmup):
            fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(args.steps):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / args.steps

    def tf(flops, ms):
        return dict(ms=round(ms, 4), tflops=round(flops / (ms * 1e-3) / 1e12, 1),
                    frac_of_bf16_peak=round(flops / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 3))

    res = {}
    for rows in (32768, 65536):
        x = to_device(I.synthetic_rows(rows, d, "bf16", seed=2), torch.bfloat16)
        y = torch.empty((rows, d), dtype=torch.bfloat16, device="cuda")
        y_lib = torch.empty_like(y)
        gu = torch.empty((rows, 2 * m), dtype=torch.bfloat16, device="cuda")
        ws = torch.empty((abi.moe_workspace_size(rows, E, 1, d, m, 1),), dtype=torch.uint8, device="cuda")
        counts = np.zeros(E, np.int64)
        counts[0] = rows
        off = torch.from_numpy(np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)).cuda()
        f_all, f_gu, f_dn = 6.0 * rows * d * m, 4.0 * rows * d * m, 2.0 * rows * d * m
        ms_ffn = timed(lambda: abi.moe_expert_ffn_packed(x, off, layer.w_gate_up, layer.w_down, y, ws))
        h = torch.empty((rows, m), dtype=torch.bfloat16, device="cuda")

        def lib_swiglu():
            torch.matmul(x, wguT, out=gu)
            torch.mul(torch.nn.functional.silu(gu[:, :m]), gu[:, m:], out=h)
            torch.matmul(h, wdnT, out=y_lib)

        ms_lib = timed(lib_swiglu)
        ms_gu = timed(lambda: torch.matmul(x, wguT, out=gu))
        ms_dn = timed(lambda: torch.matmul(h, wdnT, out=y_lib))
        lib_swiglu()
        abi.moe_expert_ffn_packed(x, off, layer.w_gate_up, layer.w_down, y, ws)
        torch.cuda.synchronize()
        yf, lf = y.float(), y_lib.float()
        rel = float((yf - lf).abs().max() / lf.abs().max())
        res[str(rows)] = {
            "packed FFN, one expert (both GEMMs, SiLU*up fused)": tf(f_all, ms_ffn),
            "library SwiGLU (gate/up GEMM, SiLU*up, down GEMM)": tf(f_all, ms_lib),
            "library gate/up GEMM alone": tf(f_gu, ms_gu),
            "library down GEMM alone": tf(f_dn, ms_dn),
            "max rel diff packed vs library output": rel,
        }
        _log(f"{rows} rows: packed {ms_ffn * 1e3:.1f} us, library SwiGLU {ms_lib * 1e3:.1f} us")
        del x, y, y_lib, gu, ws, h
        torch.cuda.empty_cache()
    r32 = res["32768"]["packed FFN, one expert (both GEMMs, SiLU*up fused)"]
    ach = r32["tflops"]
    roof = {"bound": "mfma", "achieved": ach, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
            "frac": ach / PEAK_BF16_TFLOPS, "traffic": None,
            "kernel": "moe_expert_ffn_packed, 32768 rows on one expert (ffn_pingpong_kernel)"}
    return _line(
        "Expert FFN TFLOP/s with cache-resident weights, beside the vendor GEMM library on the same shapes",
        ach, "TFLOP/s", args, r32["ms"],
        {"workload": "one expert of the Qwen3-VL-MoE layer (d 2048, m 768, bf16) at 32768 and 65536 rows; "
                     "the library leg is torch.matmul on the same operands plus torch's SiLU and product",
         "seed": 2}, roof, None, cases=res)


if __name__ == "__main__":
    sys.exit(main())
