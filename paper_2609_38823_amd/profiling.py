"""Memory traffic and MFMA counters of the dense MoE layer from rocprofv3
counter passes.

Two `rocprofv3 --pmc` passes over `bench.py --traffic-run` (one with
FETCH_SIZE, one with WRITE_SIZE; the counters of one pass must fit the
hardware) record, per dispatch, the KiB the L2 fetched from and wrote to
memory.  The same run copies a known number of bytes with
drop_visual_block (a plain row copy: N bytes read, N written), which gives
the factor between what the counter reads and the bytes actually moved.
An optional third pass (SQ_VALU_MFMA_BUSY_CYCLES, GRBM_GUI_ACTIVE,
SQ_INSTS_VALU_MFMA_MOPS_BF16) gives the expert GEMM's MFMA work and
busy cycles.

    python -m paper_2609_38823_amd.profiling FETCH_DIR WRITE_DIR OUT_PREFIX [MFMA_DIR]
    python -m paper_2609_38823_amd.profiling trace TRACE_DIR PREFIX OUT HEADER...

writes OUT_PREFIX.json (read by bench.py) and OUT_PREFIX.txt: the expert
FFN's bytes per call and, per stage of the dense span at 4096 rows
(routing, dispatch, expert FFN, combine), bytes moved, the dispatch's own
duration in the counter run and the achieved GB/s against the 8 TB/s peak.
The JSON records a hash of the GEMM sources; bench.py reports the traffic
only while the sources still hash the same.
"""

from __future__ import annotations

import collections
import csv
import glob
import hashlib
import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
KERNEL_SOURCES = ("csrc/ffn.hip", "csrc/common.hpp")
COPY_BYTES = 65536 * 2048 * 2  # the --traffic-run copy: 65536 bf16 rows of 2048


def source_hash() -> str:
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(HERE, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def _short(name: str) -> str:
    name = name.replace("decomoe::(anonymous namespace)::", "").replace("decomoe::kern::", "")
    name = name.replace("void ", "")
    out, depth = "", 0
    for ch in name:
        if ch == "(" and out.count("<") == out.count(">"):
            break
        out += ch
    return out


def per_kernel(pass_dir: str, counter: str) -> dict:
    """Mean counter value (KiB per dispatch) by (kernel, grid size)."""
    vals = collections.defaultdict(list)
    for f in glob.glob(os.path.join(pass_dir, "**", "*counter_collection.csv"), recursive=True):
        for r in csv.DictReader(open(f)):
            if r["Counter_Name"] == counter:
                vals[(_short(r["Kernel_Name"]), int(r["Grid_Size"]))].append(float(r["Counter_Value"]))
    return {k: sum(v) / len(v) for k, v in vals.items()}


def per_kernel_time(pass_dir: str) -> dict:
    """Mean dispatch duration (s) by (kernel, grid size) in a counter run."""
    vals = collections.defaultdict(list)
    seen = set()
    for f in glob.glob(os.path.join(pass_dir, "**", "*counter_collection.csv"), recursive=True):
        for r in csv.DictReader(open(f)):
            key = (r["Dispatch_Id"], r["Kernel_Name"])
            if key in seen:
                continue
            seen.add(key)
            dt = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-9
            vals[(_short(r["Kernel_Name"]), int(r["Grid_Size"]))].append(dt)
    return {k: sum(v) / len(v) for k, v in vals.items()}


PEAK_HBM = 8.0e12       # B/s
PEAK_BF16 = 2.5e15      # FLOP/s, dense
CLOCK = 2.4e9           # Hz, peak engine clock
N_SIMD = 256 * 4
N_XCC = 8

# kernels of the dense span at 4096 rows (the --traffic-run layer call)
# the persistent expert FFN at 128-row token tiles: the alternating-wavefront
# kernel where 512 divides both weight matrices, else the two-workgroup one
FFN128 = ("ffn_pingpong_kernel", "ffn_fused_kernel<128")

STAGES = [
    ("routing", [("router_x3_kernel<", None), ("topk_row_kernel<", None), ("topk_kernel<2>", 262144)]),
    ("dispatch", [("dispatch_hist_kernel", None), ("dispatch_scan_rank_kernel", None), ("dispatch_scan_kernel", None),
                  ("dispatch_rank_kernel", None)]),
    ("expert FFN", [("clear_kernel", None)] + [(k, None) for k in FFN128]),
    ("combine", [("combine_kernel<true, false", 1048576)]),
]


def stage_table(fetch, write, times, f_scale, w_scale) -> list:
    rows = []
    for label, kernels in STAGES:
        fb = wb = sec = 0.0
        names = []
        for prefix, grid in kernels:
            keys = [k for k in fetch if k[0].startswith(prefix) and (grid is None or k[1] == grid)]
            if not keys:
                continue
            key = max(keys, key=lambda k: k[1])
            fb += fetch[key] * 1024.0 * f_scale
            wb += write.get(key, 0.0) * 1024.0 * w_scale
            sec += times.get(key, 0.0)
            names.append(f"{key[0]}[{key[1]}]")
        if sec > 0:
            gbs = (fb + wb) / sec
            rows.append(dict(stage=label, kernels=names, read_bytes=fb, write_bytes=wb, seconds=sec,
                             gb_per_s=gbs / 1e9, hbm_frac=gbs / PEAK_HBM))
    return rows


def mfma_summary(mfma_dir: str) -> dict | None:
    vals = collections.defaultdict(list)
    for f in glob.glob(os.path.join(mfma_dir, "**", "*counter_collection.csv"), recursive=True):
        for r in csv.DictReader(open(f)):
            if _short(r["Kernel_Name"]).startswith(FFN128):
                name = _short(r["Kernel_Name"])
                vals[r["Counter_Name"]].append(float(r["Counter_Value"]))
    times = [v for (n, g), v in per_kernel_time(mfma_dir).items() if n.startswith(FFN128)]
    if not vals or not times:
        return None
    mops = sum(vals["SQ_INSTS_VALU_MFMA_MOPS_BF16"]) / len(vals["SQ_INSTS_VALU_MFMA_MOPS_BF16"])
    busy = sum(vals["SQ_VALU_MFMA_BUSY_CYCLES"]) / len(vals["SQ_VALU_MFMA_BUSY_CYCLES"])
    gui = sum(vals["GRBM_GUI_ACTIVE"]) / len(vals["GRBM_GUI_ACTIVE"])
    sec = times[0]
    return dict(kernel=f"{name} @ 4096 rows", mfma_flops_executed=mops * 512,
                mfma_busy_cycles_sum=busy, grbm_gui_active_sum=gui, seconds=sec,
                # busy cycles per SIMD over the kernel's duration at the peak clock
                mfma_busy_frac_at_peak_clock=busy / N_SIMD / (sec * CLOCK),
                # rocprof's MfmaUtil: busy / (GRBM_GUI_ACTIVE of one XCC x SIMDs)
                mfma_util_rocprof=busy / (gui / N_XCC * N_SIMD),
                executed_tflops=mops * 512 / sec / 1e12)


def main(argv) -> int:
    fetch_dir, write_dir, out = argv[:3]
    mfma_dir = argv[3] if len(argv) > 3 else None
    fetch = per_kernel(fetch_dir, "FETCH_SIZE")
    write = per_kernel(write_dir, "WRITE_SIZE")
    copy_key = max((k for k in fetch if k[0].startswith("drop_rows_kernel")), key=lambda k: k[1])
    f_scale = COPY_BYTES / (fetch[copy_key] * 1024.0)
    w_scale = COPY_BYTES / (write[copy_key] * 1024.0)
    # the bench's FFN call at 4096 rows (128-row tiles): one persistent launch
    # running both GEMMs, or, where it is not used, the largest grids of the
    # two per-GEMM launches
    fused = [k for k in fetch if k[0].startswith(FFN128)]
    if fused:
        keys = [max(fused, key=lambda k: k[1])]
    else:
        per_mode = {}
        for name, grid in (k for k in fetch if k[0].startswith("ffn_gemm_packed_kernel")):
            mode = name.split("<")[1].split(",")[0]
            if mode not in per_mode or grid > per_mode[mode][1]:
                per_mode[mode] = (name, grid)
        keys = [per_mode[mode] for mode in sorted(per_mode)]
    rows, total = [], 0.0
    for key in keys:
        fb = fetch[key] * 1024.0 * f_scale
        wb = write.get(key, 0.0) * 1024.0 * w_scale
        total += fb + wb
        rows.append(dict(kernel=key[0], grid=key[1], fetch_bytes=fb, write_bytes=wb,
                         fetch_kib_raw=fetch[key], write_kib_raw=write.get(key, 0.0)))
    stages = stage_table(fetch, write, per_kernel_time(fetch_dir), f_scale, w_scale)
    mfma = mfma_summary(mfma_dir) if mfma_dir else None
    res = dict(source_sha256=source_hash(), copy_bytes=COPY_BYTES,
               copy_fetch_kib_raw=fetch[copy_key], copy_write_kib_raw=write[copy_key],
               fetch_scale=f_scale, write_scale=w_scale, kernels=rows, traffic_bytes_per_call=total,
               stages=stages, mfma=mfma)
    with open(out + ".json", "w") as f:
        json.dump(res, f, indent=1)
    with open(out + ".txt", "w") as f:
        f.write("# L2<->fabric traffic (HBM plus memory-side cache hits) of moe_expert_ffn_packed_gather"
                " @ 4096 rows (Qwen3-VL-MoE layer), per call\n")
        fd, wd = os.path.relpath(fetch_dir), os.path.relpath(write_dir)
        md = os.path.relpath(mfma_dir) if mfma_dir else None
        f.write("# commands (from the repository root R, one pass each):\n")
        f.write(f"#   cd /tmp && rocprofv3 --pmc FETCH_SIZE --output-format csv -d $R/{fd} -o p"
                " -- python3 $R/bench.py --traffic-run\n")
        f.write(f"#   cd /tmp && rocprofv3 --pmc WRITE_SIZE --output-format csv -d $R/{wd} -o p"
                " -- python3 $R/bench.py --traffic-run\n")
        f.write(f"#   python -m paper_2609_38823_amd.profiling {fd} {wd} "
                + os.path.relpath(out) + (f" {md}" if md else "") + "\n")
        f.write(f"# copy calibration: drop_visual_block of {COPY_BYTES} B: FETCH_SIZE {fetch[copy_key]:.0f} KiB,"
                f" WRITE_SIZE {write[copy_key]:.0f} KiB -> scale fetch {f_scale:.3f}, write {w_scale:.3f}\n")
        for r in rows:
            f.write(f"{r['kernel']:40s} grid {r['grid']:8d}  fetch {r['fetch_bytes'] / 1e6:9.1f} MB"
                    f"  write {r['write_bytes'] / 1e6:9.1f} MB  (raw {r['fetch_kib_raw']:.0f} / "
                    f"{r['write_kib_raw']:.0f} KiB)\n")
        f.write(f"total per moe_expert_ffn_packed_gather call: {total / 1e6:.1f} MB\n")
        f.write("\n# per stage of the dense span at 4096 rows: L2<->fabric bytes (scaled), the dispatches'\n"
                "# durations in the FETCH_SIZE run, achieved GB/s against the 8 TB/s HBM peak\n")
        for r in stages:
            f.write(f"{r['stage']:12s} read {r['read_bytes'] / 1e6:8.1f} MB  write {r['write_bytes'] / 1e6:7.1f} MB"
                    f"  {r['seconds'] * 1e6:7.1f} us  {r['gb_per_s']:7.0f} GB/s  ({r['hbm_frac']:.2f} of peak)"
                    f"  {', '.join(r['kernels'])}\n")
        if mfma:
            f.write("\n# expert GEMM MFMA counters (pass: SQ_VALU_MFMA_BUSY_CYCLES GRBM_GUI_ACTIVE "
                    "SQ_INSTS_VALU_MFMA_MOPS_BF16)\n")
            f.write(f"#   cd /tmp && rocprofv3 --pmc SQ_VALU_MFMA_BUSY_CYCLES GRBM_GUI_ACTIVE "
                    f"SQ_INSTS_VALU_MFMA_MOPS_BF16 --output-format csv -d $R/{md} -o p -- "
                    f"python3 $R/bench.py --traffic-run\n")
            f.write(f"{mfma['kernel']}: {mfma['mfma_flops_executed'] / 1e9:.1f} GFLOP of bf16 MFMA executed "
                    f"(309.2 algorithmic: the rest is 32-row padding) in {mfma['seconds'] * 1e6:.1f} us = "
                    f"{mfma['executed_tflops']:.0f} TFLOP/s; MFMA busy {mfma['mfma_busy_frac_at_peak_clock']:.2f} "
                    f"of the kernel's time at 2.4 GHz; rocprof MfmaUtil (busy / GRBM_GUI_ACTIVE per XCC / "
                    f"SIMDs) {mfma['mfma_util_rocprof']:.2f}\n")
    print(open(out + ".txt").read())
    return 0


def trace_summary(argv) -> int:
    """trace TRACE_DIR PREFIX OUT HEADER_LINE...: per (kernel, grid) call
    counts and durations from a `rocprofv3 --kernel-trace --stats
    --output-format csv -o PREFIX` run, then the --stats table; the header
    lines (what ran, the command) come first."""
    trace_dir, prefix, out, header = argv[0], argv[1], argv[2], argv[3:]
    vals = collections.defaultdict(list)
    for r in csv.DictReader(open(os.path.join(trace_dir, f"{prefix}_kernel_trace.csv"))):
        vals[(_short(r["Kernel_Name"]), int(r["Grid_Size_X"]), int(r["Workgroup_Size_X"]))].append(
            (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    lines = list(header) + ["", f"## per kernel and grid (from {prefix}_kernel_trace.csv; durations in us)",
                            f"# {'kernel':58s} {'grid(thr)':>10s} {'wg':>4s} {'calls':>5s} {'avg_us':>9s}"
                            f" {'min_us':>9s} {'max_us':>9s}"]
    for (n, g, w), v in sorted(vals.items(), key=lambda kv: -sum(kv[1])):
        lines.append(f"{n[:60]:60s} {g:10d} {w:4d} {len(v):5d} {sum(v) / len(v):9.2f} {min(v):9.2f} {max(v):9.2f}")
    lines += ["", f"## rocprofv3 --stats ({prefix}_kernel_stats.csv: all launches of a kernel, every grid size)",
              f"{'kernel':60s} {'calls':>7s} {'avg_us':>9s} {'pct':>6s}"]
    for r in csv.DictReader(open(os.path.join(trace_dir, f"{prefix}_kernel_stats.csv"))):
        lines.append(f"{_short(r['Name'])[:60]:60s} {int(r['Calls']):7d} {float(r['AverageNs']) / 1e3:9.2f}"
                     f" {float(r['Percentage']):6.2f}")
    with open(out, "w") as f:
        f.write("\n".join(lines) + "\n")
    return 0


if __name__ == "__main__":
    if sys.argv[1:2] == ["trace"]:
        sys.exit(trace_summary(sys.argv[2:]))
    sys.exit(main(sys.argv[1:]))
