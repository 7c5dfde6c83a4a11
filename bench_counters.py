"""Summarises rocprofv3 runs of bench.py into the text summaries kept with the
benchmark: per-kernel timings, and HBM traffic of the grouped gate/up GEMM.

Input runs (CSV output, `-o run`), each with bench.py's --launch-log and
--phase-steps 0 (no per-phase pass after the timed steps, so that the last
gate/up dispatches are the timed ones):
  trace  rocprofv3 --kernel-trace --stats   -- python3 bench.py --phase-steps 0
  fetch  rocprofv3 --pmc FETCH_SIZE         -- python3 bench.py --phase-steps 0 --calibration --no-cpu-baseline
  write  rocprofv3 --pmc WRITE_SIZE         -- python3 bench.py --phase-steps 0 --calibration --no-cpu-baseline

`--calibration` runs torch's negation over 64 Mi fp32 (256 MiB read, 256 MiB
written) between the warm-up and the timed steps. Its counter readings give
the scale from counter KiB to bytes, and its position in dispatch order marks
where the timed steps begin: the gate/up GEMM dispatches after it are the
ones bench.py times.

The gate/up GEMM is the k_ffn instance with UP = true (hit and miss launches
use the same instance). The launch log lists the timed gate/up launches in
dispatch order with the bytes each moved host-to-device; like bench.py's
roofline, the summaries take the launches that moved none (a launch that
transfers miss weights runs as long as its PCIe reads). Traffic per launch is
the mean over those dispatches of scaled FETCH_SIZE + WRITE_SIZE.
"""
from __future__ import annotations

import argparse
import csv
import hashlib
import json
import os
import re

ROOT = os.path.dirname(os.path.abspath(__file__))
FFN_SOURCE = os.path.join(ROOT, "paper_2609_33385_amd", "csrc", "ffn.hip")
CAL_BYTES = 64 * 2 ** 20 * 4     # bytes read, and bytes written, by the calibration kernel


def is_up(name: str) -> bool:
    return "k_ffn<" in name and ", true," in name


def short(name: str) -> str:
    m = re.search(r"oled::\(anonymous namespace\)::(k_\w+)(<[^>]*>)?", name)
    if m:
        s = m.group(1) + (m.group(2) or "")
        return s.replace("oled::(anonymous namespace)::", "")
    if name.startswith("__amd_rocclr"):
        return name
    m = re.search(r"at::native::(?:\(anonymous namespace\)::)?(\w+)", name)
    return ("torch " + m.group(1)) if m else name[:60]


def read_csv(d: str, kind: str):
    path = os.path.join(d, f"run_{kind}.csv")
    with open(path) as f:
        return list(csv.DictReader(f))


def last_json_line(path: str) -> dict:
    with open(path) as f:
        lines = [ln for ln in f.read().splitlines() if ln.startswith("{")]
    return json.loads(lines[-1])


def load_log(path: str):
    with open(path) as f:
        return json.load(f)["ffn_up"]


def select(dispatches, log):
    """The dispatches of the timed launches that moved no miss weights."""
    if len(dispatches) != len(log):
        raise SystemExit(f"{len(dispatches)} gate/up dispatches, launch log has {len(log)}")
    return [d for d, (_, h2d) in zip(dispatches, log) if h2d <= 0]


def summarise_trace(d: str, bench: dict, plain: dict, log, cmd: str) -> str:
    stats = read_csv(d, "kernel_stats")
    trace = read_csv(d, "kernel_trace")
    up = sorted((r for r in trace if is_up(r["Kernel_Name"])), key=lambda r: int(r["Dispatch_Id"]))
    timed = select(up[-len(log):], log)
    n_timed = bench["roofline"]["launches"]
    if len(timed) != n_timed:
        raise SystemExit(f"{len(timed)} launches without transfer, bench.py timed {n_timed}")
    dur = [(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3 for r in timed]
    timed_avg = sum(dur) / len(dur)
    up_stats = [r for r in stats if is_up(r["Name"])][0]
    lines = [
        "# Kernel timings: bench.py default run (block-MoE layer stack, 40% residency)",
        "",
        "Workload: bf16, hidden 2048, 64 experts, top-8, intermediate 1024, 16 layers, "
        "32 tokens per iteration, cache 26/64 per layer; 8 warm-up + 64 timed steps.",
        "",
        "Command (from the repository root, `TMPDIR=/tmp`):",
        "",
        f"    {cmd}",
        "",
        f"bench.py line of this run: value {bench['value']} {bench['unit']}, "
        f"{bench['ms_per_step']} ms/step; gate/up GEMM avg_launch_us "
        f"{bench['roofline']['avg_launch_us']} over {n_timed} launches (HIP events).",
        "",
        f"`python3 bench.py` without the profiler, same machine and tree, just before: value "
        f"{plain['value']} {plain['unit']}, {plain['ms_per_step']} ms/step, gate/up GEMM "
        f"avg_launch_us {plain['roofline']['avg_launch_us']} over "
        f"{plain['roofline']['launches']} launches, roofline frac {plain['roofline']['frac']}.",
        "",
        "Under the kernel tracer the HIP events attached to each GEMM dispatch also span the "
        "tracer's own per-dispatch work, so the event figure of the profiled run is above the "
        "trace; the unprofiled run's events are the figure bench.py reports.",
        "",
        "## Gate/up GEMM (k_ffn UP=true), trace vs. bench.py events",
        "",
        "| source | launches | avg us |",
        "|---|---|---|",
        f"| rocprofv3 stats, all dispatches | {up_stats['Calls']} | "
        f"{float(up_stats['AverageNs']) / 1e3:.2f} |",
        f"| rocprofv3 trace, timed dispatches that moved no miss weights | {len(timed)} | "
        f"{timed_avg:.2f} |",
        f"| bench.py HIP events, timed steps, profiled run | {n_timed} | "
        f"{bench['roofline']['avg_launch_us']} |",
        f"| bench.py HIP events, timed steps, unprofiled run | {plain['roofline']['launches']} | "
        f"{plain['roofline']['avg_launch_us']} |",
        "",
        "## All kernels (rocprofv3 --stats)",
        "",
        "| kernel | calls | avg us | total ms | % |",
        "|---|---|---|---|---|",
    ]
    for r in stats:
        lines.append(f"| `{short(r['Name'])}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                     f"{float(r['TotalDurationNs']) / 1e6:.2f} | {float(r['Percentage']):.2f} |")
    return "\n".join(lines) + "\n"


def counter_rows(d: str, counter: str):
    rows = [r for r in read_csv(d, "counter_collection") if r["Counter_Name"] == counter]
    rows.sort(key=lambda r: int(r["Dispatch_Id"]))
    return rows


def split_timed(rows, bench: dict, log):
    cal = [i for i, r in enumerate(rows) if "neg_kernel" in r["Kernel_Name"]]
    if not cal:
        raise SystemExit("no calibration dispatch (torch neg) in the counter run")
    cal_val = float(rows[cal[-1]]["Counter_Value"])
    up = [float(r["Counter_Value"]) for r in rows[cal[-1] + 1:] if is_up(r["Kernel_Name"])]
    up = select(up, log)
    if len(up) != bench["roofline"]["launches"]:
        raise SystemExit(f"{len(up)} gate/up dispatches without transfer after calibration, "
                         f"bench.py timed {bench['roofline']['launches']}")
    return cal_val, up


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--trace", required=True, help="rocprofv3 output dir of the kernel-trace run")
    ap.add_argument("--trace-bench", required=True, help="bench.py output of the kernel-trace run")
    ap.add_argument("--trace-log", required=True, help="its --launch-log file")
    ap.add_argument("--fetch-log", required=True)
    ap.add_argument("--write-log", required=True)
    ap.add_argument("--plain-bench", required=True, help="bench.py output without the profiler")
    ap.add_argument("--fetch", required=True, help="rocprofv3 output dir of the FETCH_SIZE run")
    ap.add_argument("--fetch-bench", required=True)
    ap.add_argument("--write", required=True, help="rocprofv3 output dir of the WRITE_SIZE run")
    ap.add_argument("--write-bench", required=True)
    ap.add_argument("--out", default=os.path.join(ROOT, "profiles"))
    args = ap.parse_args()

    trace_cmd = ("rocprofv3 --kernel-trace --stats --output-format csv -d <dir> -o run "
                 "-- python3 bench.py --phase-steps 0 --launch-log <dir>/launches.json")
    tb = last_json_line(args.trace_bench)
    with open(os.path.join(args.out, "k_ffn_up_llada40_kernel_stats.md"), "w") as f:
        f.write(summarise_trace(args.trace, tb, last_json_line(args.plain_bench),
                                load_log(args.trace_log), trace_cmd))

    fb, wb = last_json_line(args.fetch_bench), last_json_line(args.write_bench)
    cal_f, up_f = split_timed(counter_rows(args.fetch, "FETCH_SIZE"), fb, load_log(args.fetch_log))
    cal_w, up_w = split_timed(counter_rows(args.write, "WRITE_SIZE"), wb, load_log(args.write_log))
    sf, sw = CAL_BYTES / cal_f, CAL_BYTES / cal_w       # bytes per counter KiB
    fetch_b = sum(up_f) / len(up_f) * sf
    write_b = sum(up_w) / len(up_w) * sw
    alg = fb["roofline"]["bytes_per_launch"]
    with open(FFN_SOURCE, "rb") as f:
        sha = hashlib.sha256(f.read()).hexdigest()
    pmc_cmd = ("timeout -s KILL 150 rocprofv3 --pmc {c} --output-format csv -d <dir> -o run "
               "-- python3 bench.py --phase-steps 0 --calibration --no-cpu-baseline "
               "--launch-log <dir>/launches.json")
    rec = {
        "kernel": "k_ffn UP=true (grouped gate/up SwiGLU GEMM)",
        "workload": "bf16 H2048 E64 k8 I1024, 16 layers, 32 tokens/iteration, cache 26/64",
        "ffn_source_sha256": sha,
        "traffic_bytes_per_launch": int(round(fetch_b + write_b)),
        "fetch_bytes_per_launch": int(round(fetch_b)),
        "write_bytes_per_launch": int(round(write_b)),
        "algorithmic_bytes_per_launch": alg,
        "launches": len(up_f),
        "fetch_scale_bytes_per_kib": sf,
        "write_scale_bytes_per_kib": sw,
        "calibration": "torch neg over 64 Mi fp32: 256 MiB read + 256 MiB written",
        "calibration_fetch_kib": cal_f,
        "calibration_write_kib": cal_w,
        "commands": [pmc_cmd.format(c="FETCH_SIZE"), pmc_cmd.format(c="WRITE_SIZE")],
    }
    with open(os.path.join(args.out, "k_ffn_up_llada40_traffic.json"), "w") as f:
        json.dump(rec, f, indent=1)
        f.write("\n")
    md = [
        "# HBM traffic: gate/up GEMM (k_ffn UP=true), block-MoE layer stack at 40% residency",
        "",
        "Commands (from the repository root, `TMPDIR=/tmp`), one counter per run:",
        "",
        *[f"    {c}" for c in rec["commands"]],
        "",
        "Scale: the calibration kernel (torch neg over 64 Mi fp32, 256 MiB read and 256 MiB "
        f"written) read FETCH_SIZE {cal_f:.0f} KiB and WRITE_SIZE {cal_w:.0f} KiB, so one "
        f"counter KiB is {sf:.1f} B fetched and {sw:.1f} B written.",
        "",
        f"Over the {len(up_f)} timed gate/up launches that moved no miss weights (hit and miss "
        "launches, dispatches after the calibration kernel):",
        "",
        "| per launch | bytes |",
        "|---|---|",
        f"| fetched (scaled FETCH_SIZE) | {fetch_b:.0f} |",
        f"| written (scaled WRITE_SIZE) | {write_b:.0f} |",
        f"| traffic | {fetch_b + write_b:.0f} |",
        f"| algorithmic (weights + activations + outputs) | {alg} |",
        f"| traffic / algorithmic | {(fetch_b + write_b) / alg:.3f} |",
        "",
        f"Kernel source sha256 `{sha}`; bench.py reports this traffic only while "
        "ffn.hip is unchanged.",
    ]
    with open(os.path.join(args.out, "k_ffn_up_llada40_traffic.md"), "w") as f:
        f.write("\n".join(md) + "\n")
    print(json.dumps({k: rec[k] for k in ("traffic_bytes_per_launch", "algorithmic_bytes_per_launch",
                                          "launches")}))


if __name__ == "__main__":
    main()
