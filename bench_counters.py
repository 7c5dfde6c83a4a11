"""Summarises rocprofv3 runs of bench.py into the text summaries kept under
profiles/: the kernel trace of the timed steps against bench.py's own HIP
events, HBM traffic of the grouped GEMM launches from hardware counters
against their algorithmic bytes, and matrix-core busy cycles.

Input runs (CSV output, `-o run`), each of the same bench.py command with
--phase-steps 0 --full-steps 0 --no-secondary --no-cpu-baseline --calibration
--launch-log <dir>/launches.json --profile-ops ffn_up,ffn_down,ffn_dense_up,ffn_dense_down
and the workload's own flags:
  trace  rocprofv3 --kernel-trace --stats
  fetch  rocprofv3 --pmc FETCH_SIZE
  write  rocprofv3 --pmc WRITE_SIZE
  mfma   rocprofv3 --pmc SQ_VALU_MFMA_BUSY_CYCLES SQ_BUSY_CYCLES GRBM_GUI_ACTIVE

`--calibration` runs torch's negation over 64 Mi fp32 (256 MiB read, 256 MiB
written) between the warm-up and the timed steps: its counter readings give
the scale from counter KiB to bytes, and its position in dispatch order marks
where the timed steps begin. The launch log lists the timed operations in
order with their algorithmic bytes, flops and host-to-device bytes; the
dispatches of each GEMM kernel after the calibration kernel are matched to
them in order:
  k_ffn<..., true, ...>   gate/up GEMM of the cached experts (+ the misses'
                          gate/up copy)                       <- ffn_up
  k_ffn_mix<...>          cached experts' down GEMM + the misses' down copy
                          + the misses' gate/up GEMM          <- ffn_down, 1st of each layer
  k_ffn<..., false, ...>  the misses' down GEMM               <- ffn_down, 2nd of each layer
  k_ffn_dense<true/false> dense tiles                        <- ffn_dense_up / _down
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
N_SIMD = 1024                    # 256 CUs x 4 SIMDs
N_XCD = 8                        # GRBM_GUI_ACTIVE sums the busy cycles of the 8 XCDs
CLASSES = ("up", "mix", "down", "dense_up", "dense_down")
MIN_CLOCK_NS = 200_000           # clock column only for dispatches of 200 us or more


def kclass(name: str):
    if "k_ffn_mix<" in name:
        return "mix"
    if "k_ffn_dense<true>" in name:
        return "dense_up"
    if "k_ffn_dense<false>" in name:
        return "dense_down"
    if "k_ffn<" in name:
        return "up" if ", true," in name else "down"
    return None


def short(name: str) -> str:
    m = re.search(r"oled::\(anonymous namespace\)::(k_\w+)(<[^>]*>)?", name)
    if m:
        return m.group(1) + (m.group(2) or "")
    if name.startswith("__amd_rocclr"):
        return name
    m = re.search(r"at::native::(?:\(anonymous namespace\)::)?(\w+)", name)
    return ("torch " + m.group(1)) if m else name[:60]


def read_csv(d: str, kind: str):
    with open(os.path.join(d, f"run_{kind}.csv")) as f:
        return list(csv.DictReader(f))


def last_json_line(path: str) -> dict:
    with open(path) as f:
        lines = [ln for ln in f.read().splitlines() if ln.startswith("{")]
    return json.loads(lines[-1])


def ops_by_class(log_path: str):
    """The timed operations of the launch log per kernel class, in order."""
    with open(log_path) as f:
        ops = json.load(f)["ops"]
    down = [o for o in ops if o[0] == "ffn_down"]
    return {"up": [o for o in ops if o[0] == "ffn_up"], "mix": down[0::2], "down": down[1::2],
            "dense_up": [o for o in ops if o[0] == "ffn_dense_up"],
            "dense_down": [o for o in ops if o[0] == "ffn_dense_down"]}


def timed_dispatches(rows, key="Dispatch_Id"):
    """Rows after the last calibration dispatch, per kernel class, in order."""
    rows = sorted(rows, key=lambda r: int(r[key]))
    cal = [i for i, r in enumerate(rows) if "neg_kernel" in r["Kernel_Name"]]
    if not cal:
        raise SystemExit("no calibration dispatch (torch neg) in the run")
    out = {c: [] for c in CLASSES}
    for r in rows[cal[-1] + 1:]:
        c = kclass(r["Kernel_Name"])
        if c:
            out[c].append(r)
    return rows[cal[-1]], out


def counter_run(d: str, counter: str, ops):
    rows = [r for r in read_csv(d, "counter_collection") if r["Counter_Name"] == counter]
    cal, per = timed_dispatches(rows)
    for c in CLASSES:
        if len(per[c]) != len(ops[c]):
            raise SystemExit(f"{counter}: {len(per[c])} {c} dispatches after calibration, "
                             f"launch log has {len(ops[c])}")
    return float(cal["Counter_Value"]), {c: [float(r["Counter_Value"]) for r in per[c]]
                                         for c in CLASSES}


def mean(v):
    return sum(v) / len(v) if v else 0.0


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--name", required=True, help="workload tag of the summaries (e128_zipf40)")
    ap.add_argument("--workload-text", required=True)
    ap.add_argument("--command", required=True, help="the bench.py command line of the runs")
    ap.add_argument("--plain-bench", required=True, help="bench.py output without the profiler")
    for run in ("trace", "fetch", "write", "mfma"):
        ap.add_argument(f"--{run}", required=True, help=f"rocprofv3 output dir of the {run} run")
        ap.add_argument(f"--{run}-bench", required=True)
        ap.add_argument(f"--{run}-log", required=True)
    ap.add_argument("--out", default=os.path.join(ROOT, "profiles"))
    args = ap.parse_args()
    plain = last_json_line(args.plain_bench)

    # ---- kernel trace against the events
    tb = last_json_line(args.trace_bench)
    ops_t = ops_by_class(args.trace_log)
    trace = read_csv(args.trace, "kernel_trace")
    _, per_t = timed_dispatches(trace)
    if len(per_t["up"]) != len(ops_t["up"]):
        raise SystemExit(f"trace: {len(per_t['up'])} gate/up dispatches, log {len(ops_t['up'])}")
    dur = {c: [(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3 for r in per_t[c]]
           for c in CLASSES}
    ev = {c: [o[2] * 1e3 for o in ops_t[c]] for c in CLASSES}
    stats = read_csv(args.trace, "kernel_stats")
    cmd_trace = f"rocprofv3 --kernel-trace --stats --output-format csv -d <dir> -o run -- {args.command}"
    md = [f"# Kernel trace: bench.py on the {args.workload_text}", "",
          "Command (repository root, `TMPDIR=/tmp`):", "", f"    {cmd_trace}", "",
          f"bench.py line of this run: value {tb['value']} {tb['unit']}, {tb['ms_per_step']} "
          f"ms per step. Without the profiler, same machine and tree: value {plain['value']} "
          f"{plain['unit']}, {plain['ms_per_step']} ms per step; gate/up GEMM "
          f"avg_launch_us {plain['roofline']['avg_launch_us']} over "
          f"{plain['roofline']['launches']} launches (HIP events on the dispatches).", "",
          "## Timed GEMM launches: trace against the HIP events of the same run", "",
          "| kernel | launches | trace avg us | events avg us |", "|---|---|---|---|"]
    for c in CLASSES:
        if dur[c]:
            md.append(f"| {c} | {len(dur[c])} | {mean(dur[c]):.2f} | {mean(ev[c]):.2f} |")
    md += ["", "## All kernels of the run (rocprofv3 --stats)", "",
           "| kernel | calls | avg us | total ms | % |", "|---|---|---|---|---|"]
    for r in stats:
        md.append(f"| `{short(r['Name'])}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                  f"{float(r['TotalDurationNs']) / 1e6:.2f} | {float(r['Percentage']):.2f} |")
    with open(os.path.join(args.out, f"k_ffn_up_{args.name}_kernel_stats.md"), "w") as f:
        f.write("\n".join(md) + "\n")

    # ---- HBM traffic per launch class
    ops_f, ops_w = ops_by_class(args.fetch_log), ops_by_class(args.write_log)
    cal_f, fetch = counter_run(args.fetch, "FETCH_SIZE", ops_f)
    cal_w, write = counter_run(args.write, "WRITE_SIZE", ops_w)
    sf, sw = CAL_BYTES / cal_f, CAL_BYTES / cal_w     # bytes per counter KiB
    ops_m = ops_by_class(args.mfma_log)
    mfma, gui, clk = {}, {}, {}
    for cnt, dst in (("SQ_VALU_MFMA_BUSY_CYCLES", mfma), ("GRBM_GUI_ACTIVE", gui)):
        rows = [r for r in read_csv(args.mfma, "counter_collection") if r["Counter_Name"] == cnt]
        _, per = timed_dispatches(rows)
        for c in CLASSES:
            dst[c] = [float(r["Counter_Value"]) for r in per[c]]
            if cnt == "GRBM_GUI_ACTIVE":   # shader-clock cycles per XCD over the dispatch
                durs = [max(1, int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) for r in per[c]]
                # the counter's window exceeds short dispatches: clock only for long ones
                clk[c] = ([float(r["Counter_Value"]) / N_XCD / d for r, d in zip(per[c], durs)]
                          if durs and mean(durs) >= MIN_CLOCK_NS else [])
    with open(FFN_SOURCE, "rb") as f:
        sha = hashlib.sha256(f.read()).hexdigest()
    rows_md, per_class = [], {}
    for c in CLASSES:
        if not ops_f[c]:
            continue
        alg = mean([o[3] for o in ops_f[c]])
        h2d = mean([max(0, o[5]) for o in ops_f[c]])
        fb, wb = mean(fetch[c]) * sf, mean(write[c]) * sw
        flops = mean([o[4] for o in ops_t[c]])
        busy = mean(mfma[c]) / (N_SIMD * mean(gui[c]) / N_XCD) if mean(gui[c]) else None
        t_us = mean([o[2] for o in ops_t[c]]) * 1e3
        flop_util = flops / (t_us * 1e-6) / 2.5e15 if t_us > 0 else None
        ghz = mean(clk[c]) if clk[c] else None
        per_class[c] = dict(launches=len(ops_f[c]), algorithmic_bytes=int(alg), h2d_bytes=int(h2d),
                            fetch_bytes=int(fb), write_bytes=int(wb), mfma_busy=busy,
                            flop_util=flop_util, clock_ghz=ghz)
        rows_md.append(f"| {c} | {len(ops_f[c])} | {alg / 1e6:.1f} | {h2d / 1e6:.1f} | "
                       f"{fb / 1e6:.1f} | {wb / 1e6:.1f} | {(fb + wb) / max(1.0, alg + 2 * h2d):.3f} | "
                       f"{'—' if ghz is None else f'{ghz:.2f}'} | {busy:.4f} | {flop_util:.4f} |")
    up = per_class["up"]
    rec = {"kernel": "k_ffn UP=true (grouped gate/up SwiGLU GEMM, with the misses' gate/up copy)",
           "workload": args.workload_text, "ffn_source_sha256": sha,
           "traffic_bytes_per_launch": up["fetch_bytes"] + up["write_bytes"],
           "fetch_bytes_per_launch": up["fetch_bytes"], "write_bytes_per_launch": up["write_bytes"],
           "algorithmic_bytes_per_launch": up["algorithmic_bytes"],
           "h2d_bytes_per_launch": up["h2d_bytes"], "launches": up["launches"],
           "fetch_scale_bytes_per_kib": sf, "write_scale_bytes_per_kib": sw,
           "calibration": "torch neg over 64 Mi fp32: 256 MiB read + 256 MiB written",
           "per_class": per_class,
           "commands": [f"timeout -s KILL 300 rocprofv3 --pmc {c} --output-format csv -d <dir> -o run "
                        f"-- {args.command}" for c in ("FETCH_SIZE", "WRITE_SIZE",
                                                      "SQ_VALU_MFMA_BUSY_CYCLES SQ_BUSY_CYCLES "
                                                      "GRBM_GUI_ACTIVE")]}
    with open(os.path.join(args.out, f"k_ffn_up_{args.name}_traffic.json"), "w") as f:
        json.dump(rec, f, indent=1)
        f.write("\n")
    md = [f"# Grouped GEMM launches: counters on the {args.workload_text}", "",
          "Commands (repository root, `TMPDIR=/tmp`), one counter set per run:", "",
          *[f"    {c}" for c in rec["commands"]], "",
          f"Scale: the calibration kernel (torch neg over 64 Mi fp32) read FETCH_SIZE {cal_f:.0f} "
          f"KiB and WRITE_SIZE {cal_w:.0f} KiB for 256 MiB each way, so one counter KiB is "
          f"{sf:.1f} B fetched and {sw:.1f} B written.", "",
          "Per launch, averaged over the timed launches of each class (MB = 1e6 bytes). "
          "Algorithmic bytes are the GEMM's own operands (weights, token rows, outputs); "
          "launches that carry the misses' copy also read those bytes from pinned host memory "
          "and write them into their slots, so the ratio's denominator adds twice the copied "
          "bytes. MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES (summed over the 1024 SIMDs) / (1024 x "
          "GRBM_GUI_ACTIVE / 8): the share of the launch's shader-clock cycles the matrix "
          "cores were busy (GRBM_GUI_ACTIVE counts shader-clock cycles summed over the 8 XCDs; "
          "divided by 8 and by the dispatch's duration it gives the clock the launch ran at, "
          "the clock column, shown for classes whose dispatches last 200 us or more: the "
          "counter's window exceeds shorter ones, which also makes their MFMA busy a lower "
          "bound); it counts the MFMAs of padded tile rows too. Flop util = "
          "algorithmic flops / event time of the trace run / 2.5 PFLOP/s.", "",
          "| launch class | launches | algorithmic MB | copied host->device MB | fetched MB | "
          "written MB | traffic / (algorithmic + 2 x copied) | clock (GHz) | MFMA busy | "
          "flop util |",
          "|---|---|---|---|---|---|---|---|---|---|", *rows_md, "",
          f"Kernel source sha256 `{sha}`; bench.py reports the gate/up traffic only while "
          "ffn.hip is unchanged."]
    with open(os.path.join(args.out, f"ffn_kernels_{args.name}_counters.md"), "w") as f:
        f.write("\n".join(md) + "\n")
    print(json.dumps({"traffic_bytes_per_launch": rec["traffic_bytes_per_launch"],
                      "per_class": per_class}))


if __name__ == "__main__":
    main()
