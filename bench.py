#!/usr/bin/env python3
"""MoE-layer throughput of the RCEP hot path on one MI355X.

One step is one prefill of the Qwen3-VL-MoE-shaped MoE layer through the
visual exit (Algorithm 2 of the paper), on synthetic inputs already
resident in HBM:

  dense span   moe_route -> moe_dispatch -> moe_expert_ffn -> moe_combine
               over 4096 rows (3584 visual + 512 text), all 128 experts
  SAVB exit    drop_visual_block removes the 3584 visual rows
  RCEP span    moe_route (full pool) -> moe_calibrate_prefix (K, p = 0.9)
               -> moe_route (prefix re-route) -> moe_dispatch
               -> moe_expert_ffn (experts [0, K)) -> moe_combine
               over the 512 text rows

value = MoE-layer tokens per second over the step (4096 + 512 rows per
step).  Every ABI call is bracketed by HIP events on the stream it runs on,
giving per-stage times and the roofline of the dominant kernel (the expert
FFN).  The CPU oracle is timed on the same step as the CPU baseline.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline]
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


def stage_flops_bytes(stage: str, T: int, d: int, E: int, m: int, k: int, touched: int, K: int):
    """Algorithmic FLOPs and HBM bytes of one ABI call (bf16 rows, fp32
    router and routing arrays).  Sizes per row and per expert are listed in
    the design notes."""
    A = T * k
    if stage == "route_full":
        return 2.0 * T * d * E, T * d * 2 + d * E * 4 + E * 4 + T * E * 4 + 2 * T * k * 4
    if stage == "route_prefix":
        return 0.0, T * K * 4 + 2 * T * k * 4
    if stage == "calibrate":
        return 0.0, 2 * T * k * 4 + E * 8 + 4
    if stage == "dispatch":
        return 0.0, T * k * 4 + (E + 1) * 8 + 2 * A * 4 + T * d * 2 + A * d * 2
    if stage == "ffn":
        return 6.0 * A * d * m, touched * 3 * d * m * 2 + 2 * A * d * 2 + (E + 1) * 4
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


def measured_traffic():
    """HBM bytes per FFN call from the committed counter passes, or None
    when the GEMM sources changed since they were taken."""
    try:
        from paper_2609_38823_amd.profiling import source_hash
        rec = json.load(open(TRAFFIC_FILE))
        if rec.get("source_sha256") != source_hash():
            return None
        return rec["traffic_bytes_per_call"]
    except (OSError, ValueError, KeyError):
        return None


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
    """The same step on the CPU oracle (test infrastructure, timed only)."""
    import oracle
    t0 = time.perf_counter()
    oracle.moe_layer_dense(x, params["w_r"], params["bias"], params["w_gate_up"], params["w_down"], k)
    h = oracle.drop_visual_block(x, 0, x.shape[0] - text.shape[0])
    oracle.moe_layer_rcep(h, params["w_r"], params["bias"], params["w_gate_up"], params["w_down"], k, p)
    return time.perf_counter() - t0


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--traffic-run", action="store_true",
                    help="only run the dense layer and a known-size copy (for rocprofv3 counter passes)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: the path has no multi-GPU execution in this build "
              "(see the design notes for how it would shard); run with --gpus 1", file=sys.stderr)
        return 2

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
    stages = ["route_full", "dispatch", "ffn", "combine", "drop",
              "r.route_full", "r.calibrate", "r.route_prefix", "r.dispatch", "r.ffn", "r.combine"]

    def step(ev=None):
        marks = iter(ev) if ev is not None else None

        def mark():
            if marks is not None:
                next(marks).record(stream)

        mark()
        layer.forward_dense(x, bd, mark=mark)
        abi.drop_visual_block(x, 0, V, h_text)
        mark()
        layer.forward_rcep(h_text, p, b=br, mark=mark)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(len(stages) + 1)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(args.steps):
        step(evs[s])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = wall * 1e3 / args.steps
    stage_ms = {}
    for i, name in enumerate(stages):
        stage_ms[name] = float(np.mean([e[i].elapsed_time(e[i + 1]) for e in evs]))

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
    rcep_ms = sum(stage_ms[s] for s in stages if s.startswith("r."))
    spans = {
        "dense@4096": dict(ms=round(dense_ms, 4), tokens_per_s=T / dense_ms * 1e3,
                           tflops=per_tok_flops * T / dense_ms / 1e9, touched_experts=touched_d),
        "rcep@512": dict(ms=round(rcep_ms, 4), tokens_per_s=(T - V) / rcep_ms * 1e3,
                         tflops=per_tok_flops * (T - V) / rcep_ms / 1e9, K=K, touched_experts=touched_r,
                         paper_dense_equiv_tflops=(2 * d * E + 6 * K * d * m) * (T - V) / rcep_ms / 1e9),
        "dense@512": dict(ms=round(dense512_ms, 4), tokens_per_s=(T - V) / dense512_ms * 1e3,
                          tflops=per_tok_flops * (T - V) / dense512_ms / 1e9, touched_experts=touched_512,
                          paper_dense_equiv_tflops=(2 * d * E + 6 * E * d * m) * (T - V) / dense512_ms / 1e9),
    }
    f, b = fb("ffn", T, touched_d)
    ffn_roof = roofline(f, b, stage_ms["ffn"] * 1e-3)
    ffn_roof["traffic"] = measured_traffic()
    ffn_roof["kernel"] = ("moe_expert_ffn_packed @ dense 4096 rows (gate/up GEMM + down GEMM launches "
                          "on packed bf16 weights)")
    ffn_roof["mfma_frac"] = f / (stage_ms["ffn"] * 1e-3) / 1e12 / PEAK_BF16_TFLOPS

    cpu = None
    if not args.no_cpu_baseline:
        sec = run_oracle_step(x_np, x_np[V:], rprm, k, p)
        info = cpu_info()
        cpu = dict(value=(T + (T - V)) / sec, unit="tokens/s",
                   cores=info.get("blas_threads") or info["affinity_cores"], kind="oracle",
                   sample="one full step (dense 4096 rows + visual drop + RCEP 512 rows), numpy float64",
                   seconds=round(sec, 3), **info)

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
        "setup_s": round(setup_s, 1),
    }
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
