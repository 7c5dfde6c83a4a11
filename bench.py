"""Block-MoE layer throughput on one MI355X under 40% expert residency.

Workload: LLaDA-MoE-like layer stack in bf16 - hidden 2048, 64 experts,
top-8, expert SwiGLU intermediate 1024, 16 MoE layers, batch 1 x block 32
tokens, 8 denoising iterations per block, expert cache 26 of 64 experts per
layer (40%). One step is one denoising iteration through all 16 layers: per
layer route_block -> moe_forward_cached (cached experts) -> apply_misses
(host-to-device copies of missed experts on a side stream, their GEMMs, the
combine) -> score_and_retain. Blocks follow each
other without resetting the caches; the warm-up steps cover the cold start.

Inputs (router logits, activations, confidence) are generated before timing
and resident in HBM; the expert weights live in a pinned host pool (all
16 x 64 experts, 12 GiB) and reach the GPU only through cache misses.

Prints one JSON line with the layer-token throughput, the roofline of the
dominant kernel (grouped gate/up GEMM, timed with HIP events on its stream
during the timed steps) and the CPU oracle timed on a bounded sample. After
the timed steps, a short pass on a second context times every operation
(detail.phase_pass: per-phase device times, their rates against HBM, and the
overlap of miss transfers with compute); it is not part of the timed region.
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

HBM_PEAK_GBS = 8000.0        # MI355X HBM3E
MFMA_BF16_PEAK_TFLOPS = 2500.0  # dense bf16 MFMA
METRIC = "block-MoE layer tokens/s at 40% expert residency; grouped-GEMM MFMA util"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def fill_pool_device(pool, w, seed: int, chunk: int = 64):
    """Fills the pinned pool with N(0, 0.02^2) bf16 weights drawn on the GPU."""
    import torch
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    host = torch.from_numpy(pool.view(np.int16))
    per = w.expert_elems
    for b0 in range(0, pool.n_blocks, chunk):
        n = min(chunk, pool.n_blocks - b0)
        v = (torch.randn(n * per, generator=g, device="cuda") * 0.02).to(torch.bfloat16)
        host[b0 * per:(b0 + n) * per].copy_(v.view(torch.int16))
    torch.cuda.synchronize()


def make_inputs(w, seed: int, n_steps: int):
    """Device tensors: logits[g][l] [T][E] fp32, x[g][l] [T][H] bf16, conf[g] [T]."""
    import torch
    from paper_2609_33385_amd import harness as HN
    from paper_2609_33385_amd import workload as W
    N, L = w.n_iters, w.n_layers
    n_blocks = (n_steps + N - 1) // N
    lg = np.empty((n_blocks * N, L, w.tokens, w.n_experts), np.float32)
    for b in range(n_blocks):
        for l in range(L):
            lg[b * N:(b + 1) * N, l] = W.logits_block(w, seed, l, b)
    xs = np.empty((n_steps, L, w.tokens, w.hidden), np.uint16)
    cf = np.empty((n_steps, w.tokens), np.float32)
    for g in range(n_steps):
        b, it = divmod(g, N)
        cf[g] = W.confidence(w, seed, b, it)
        for l in range(L):
            xs[g, l] = W.activations(w, seed, l, b, it)
    return (torch.from_numpy(lg[:n_steps]).cuda(), HN.to_device(xs), torch.from_numpy(cf).cuda())


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "k_ffn_up_llada40_traffic.json")
FFN_SOURCE = os.path.join(ROOT, "paper_2609_33385_amd", "csrc", "ffn.hip")


def measured_traffic():
    """HBM bytes per gate/up GEMM launch from the committed counter summary, or
    None if the kernel source changed since the counters were taken."""
    import hashlib
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
        with open(FFN_SOURCE, "rb") as f:
            sha = hashlib.sha256(f.read()).hexdigest()
    except (OSError, ValueError):
        return None
    if rec.get("ffn_source_sha256") != sha:
        return None
    return rec.get("traffic_bytes_per_launch")


def profile_coop(w, pool, logits, xs, conf, args):
    """Split constants of the cooperative compensation, profiled on this
    machine: T_H2D (one expert block host->device), tau_CPU (CPU expert time
    per routed token at nbar tokens) and nbar (routed tokens per missed
    expert, from a run of the warm-up steps without CPU execution)."""
    import torch
    from paper_2609_33385_amd import oled
    from paper_2609_33385_amd import workload as W
    L, T = w.n_layers, w.tokens
    ctx = oled.Context(w.hidden, w.inter, w.n_experts, w.top_k, L, w.capacity, T, w.dtype,
                       pool.ptr, pool.n_blocks, W.host_block_of(w, pool.n_blocks))
    y = torch.empty((T, w.hidden), dtype=torch.bfloat16, device="cuda")
    s = torch.cuda.current_stream()
    for g in range(args.warmup):
        for l in range(L):
            ctx.route_block(l, logits[g, l].data_ptr(), T, s)
            ctx.moe_forward_cached(l, xs[g, l].data_ptr(), y.data_ptr(), s)
            ctx.apply_misses(l, report=False)
            ctx.score_and_retain(l, conf[g].data_ptr(), s)
    st = ctx.collect_stats()
    ctx.close()
    nbar = st["n_miss_rows"] / max(1, st["n_misses"])
    # T_H2D: copy of one expert block from the pinned pool
    host = torch.from_numpy(pool.view(np.uint8)[: w.expert_bytes])
    dev = torch.empty(w.expert_bytes, dtype=torch.uint8, device="cuda")
    dev.copy_(host, non_blocking=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(20):
        dev.copy_(host, non_blocking=True)
    torch.cuda.synchronize()
    t_h2d = (time.perf_counter() - t0) / 20 * 1e6
    # tau_CPU: the CPU expert kernels on nbar tokens
    n = max(1, int(round(nbar)))
    block = pool.block(0, np.uint16)
    x = W.activations(w.replace(batch=1, block=n), args.seed, 0, 0, 0)
    oled.oled_cpu_ffn(w.dtype, w.hidden, w.inter, block, x, args.coop_threads)
    t0 = time.perf_counter()
    for _ in range(5):
        oled.oled_cpu_ffn(w.dtype, w.hidden, w.inter, block, x, args.coop_threads)
    tau = (time.perf_counter() - t0) / 5 * 1e6 / n
    lam = t_h2d if args.coop_lambda is None else args.coop_lambda
    return dict(threads=args.coop_threads, t_h2d_us=round(t_h2d, 2), tau_cpu_us=round(tau, 2),
                nbar=round(nbar, 3), lambda_us=round(lam, 2))


PHASES = ("route_topk", "permute", "ffn_up", "ffn_down", "ffn_dense_up", "ffn_dense_down",
          "h2d", "combine", "score_retain", "layer_adapt")


def pinned_h2d_gbps(pool, w):
    """Host-to-device rate of plain copies of one expert block from the pinned
    pool (hipMemcpyAsync, 20 copies)."""
    import torch
    host = torch.from_numpy(pool.view(np.uint8)[: w.expert_bytes])
    dev = torch.empty(w.expert_bytes, dtype=torch.uint8, device="cuda")
    dev.copy_(host, non_blocking=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(20):
        dev.copy_(host, non_blocking=True)
    torch.cuda.synchronize()
    return 20 * w.expert_bytes / (time.perf_counter() - t0) / 1e9


def phase_pass(w, pool, step_fn, make_ctx, args):
    """Per-phase device times, outside the timed steps: a second context with
    every operation timed (HIP events around each launch), the same warm-up,
    then args.phase_steps steps over the timed steps' inputs.

    Per phase: launches, microseconds per layer-iteration, and the rate of its
    algorithmic bytes against HBM. Overlap efficiency over the layer-iterations
    that transferred misses: sum of max(t_copy, t_compute) / sum of t_layer,
    with t_layer the device time of the layer's launches, t_copy its
    transferred bytes at the pinned host-to-device rate of plain copies, and
    t_compute the mean t_layer of the layer-iterations without transfers
    (same shapes, all work on cached experts); 1.0 means the copy hides all
    compute or the compute hides all of the copy. Shader transfer only: with
    copy-engine copies the layer's span is not the sum of its launches."""
    import torch
    from paper_2609_33385_amd import oled
    ctx = make_ctx(oled.PROFILE_ALL)
    try:
        for g in range(args.warmup):
            step_fn(ctx, g)
        torch.cuda.synchronize()
        ctx.profile_collect()
        t0 = time.perf_counter()
        for g in range(args.warmup, args.warmup + args.phase_steps):
            step_fn(ctx, g)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        ops = ctx.profile_collect()
    finally:
        ctx.close()
    groups = []
    for o in ops:                        # a layer-iteration starts with its routing
        if o[0] in ("route_topk", "route_gemm") or not groups:
            groups.append([])
        groups[-1].append(o)
    n_li = max(1, len(groups))
    phases = {}
    for name in PHASES:
        sel = [o for o in ops if o[0] == name]
        if not sel:
            continue
        ms = sum(o[2] for o in sel)
        by = sum(o[3] for o in sel)
        gbs = (by / 1e9) / (ms / 1e3) if ms > 0 else None
        phases[name] = {"launches": len(sel), "us_per_layer_iter": round(ms * 1e3 / n_li, 2),
                        "avg_us": round(ms * 1e3 / len(sel), 2),
                        "GBps": round(gbs, 1) if gbs else None,
                        "hbm_frac": round(gbs / HBM_PEAK_GBS, 4) if gbs else None}
        calm_sel = [o for o in sel if o[5] == 0]
        if name != "h2d" and 0 < len(calm_sel) < len(sel):
            # launches that also carried miss weights run as long as the PCIe reads
            cms = sum(o[2] for o in calm_sel)
            cgb = (sum(o[3] for o in calm_sel) / 1e9) / (cms / 1e3) if cms > 0 else None
            phases[name]["without_transfer"] = {
                "launches": len(calm_sel), "avg_us": round(cms * 1e3 / len(calm_sel), 2),
                "GBps": round(cgb, 1) if cgb else None,
                "hbm_frac": round(cgb / HBM_PEAK_GBS, 4) if cgb else None}
    link = pinned_h2d_gbps(pool, w)
    # launches on the compute stream (copy-engine copies run beside them)
    t_layer = [sum(o[2] for o in gr if o[0] != "h2d") for gr in groups]
    xfer = [sum(max(0, o[5]) for o in gr) for gr in groups]
    calm = [t for t, b in zip(t_layer, xfer) if b == 0]
    t_comp = float(np.mean(calm)) if calm else None
    miss = [(t, b) for t, b in zip(t_layer, xfer) if b > 0]
    overlap = None
    if miss and t_comp is not None and args.copy_mode == "shader":
        # every launch of a layer is on the compute stream, one after another,
        # so their durations add up to the layer's device time
        overlap = round(sum(max(b / (link * 1e6), t_comp) for t, b in miss)
                        / sum(t for t, b in miss), 4)
    return {"steps": args.phase_steps, "layer_iters": len(groups), "phases": phases,
            "device_busy_frac": round(sum(t_layer) / 1e3 / wall, 4) if wall > 0 else None,
            "layer_us_without_transfer": round(t_comp * 1e3, 2) if t_comp else None,
            "layer_us_with_transfer": round(float(np.mean([t for t, b in miss])) * 1e3, 2)
            if miss else None,
            "pinned_h2d_GBps": round(link, 2), "overlap_efficiency": overlap}


def cpu_baseline(w, seed: int):
    """The oracle on host cores: every layer of block 0, iterations 1-4, with the FFN."""
    from threadpoolctl import threadpool_info

    from oracle import oled_oracle as O
    from paper_2609_33385_amd import workload as W
    P = 64
    raw = {b: W.expert_block(w, seed, b) for b in range(P)}   # drawn outside the timing
    hbo = W.host_block_of(w, P)
    res0 = [np.zeros(w.n_experts, bool) for _ in range(w.n_layers)]
    for l in range(w.n_layers):                               # iteration 0 fills R (untimed)
        res0[l] = O.layer_step(W.logits(w, seed, l, 0, 0), W.confidence(w, seed, 0, 0), res0[l],
                               w.top_k, w.capacity)["resident_after"]
    iters = (1, 2, 3, 4)
    inputs = {it: (W.confidence(w, seed, 0, it),
                   [(W.logits(w, seed, l, 0, it), O.decode(W.activations(w, seed, l, 0, it)))
                    for l in range(w.n_layers)]) for it in iters}
    t0 = time.perf_counter()
    for it in iters:
        conf, rows = inputs[it]
        for l, (lg, x) in enumerate(rows):
            st = O.layer_step(lg, conf, res0[l], w.top_k, w.capacity)
            res0[l] = st["resident_after"]

            def weights(e, l=l):
                return W.split_expert(w, O.decode(raw[int(hbo[l * w.n_experts + e])]))

            O.moe_output(x, st["idx"], st["gates"], weights)
    dt = time.perf_counter() - t0
    n = len(iters) * w.n_layers
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    return {"value": n * w.tokens / dt, "unit": "layer-tokens/s", "cores": int(threads),
            "kind": "oracle",
            "sample": (f"{n} layer-iterations (all {w.n_layers} layers of block 0, iterations 1-4) "
                       f"of the same workload: routing, permutation, hit/miss sets, priorities, "
                       f"retention and the float64 SwiGLU experts + combine; {dt:.1f} s, BLAS on "
                       f"{threads} threads of {os.cpu_count()} host CPUs")}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=64)
    ap.add_argument("--warmup", type=int, default=8)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--capacity", type=int, default=None, help="experts cached per layer")
    ap.add_argument("--workload", type=int, default=2, choices=[2, 3, 4, 5],
                    help="2: the 40%% stack with 32 tokens per iteration (the headline); 3: the "
                         "same stack with batch 8 x block 32 = 256 tokens per iteration; 4: the "
                         "E=128 stack (hidden 4096, 48 layers, 1024 tokens, Zipf popularity, "
                         "40%%); 5: its stress form (20%%, iteration noise 1.5). 4 and 5 alias "
                         "their experts onto --pool-blocks host blocks and take minutes per "
                         "few steps: pass small --warmup/--steps")
    ap.add_argument("--pool-blocks", type=int, default=None,
                    help="distinct pinned host blocks (default: every expert, up to 16 GiB)")
    ap.add_argument("--adapt-period", type=int, default=0,
                    help="layer-adaptive cache sizing every N iterations (0: fixed capacity "
                         "per layer, the headline configuration)")
    ap.add_argument("--coop", action="store_true",
                    help="cooperative compensation (CPU execution of part of the misses); its "
                         "split constants are profiled here before the timed steps")
    ap.add_argument("--coop-threads", type=int, default=8)
    ap.add_argument("--coop-lambda", type=float, default=None,
                    help="lambda in microseconds per unit of priority (default: T_H2D)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--phase-steps", type=int, default=8,
                    help="after the timed steps, this many steps on a second context with every "
                         "operation timed: per-phase times and overlap efficiency (0: skip)")
    ap.add_argument("--calibration", action="store_true",
                    help="between warm-up and timed steps, run a plain streaming kernel of known traffic (torch "
                         "negation over 256 MiB fp32: 256 MiB read, 256 MiB written) to scale "
                         "hardware byte counters")
    ap.add_argument("--copy-mode", default="shader", choices=["shader", "sdma"],
                    help="transfer of the misses: workgroups of the hit GEMM launches (shader) "
                         "or hipMemcpyAsync on a copy stream (sdma)")
    ap.add_argument("--launch-log", default=None,
                    help="write the timed gate/up launches in order ([bytes, h2d bytes] each) "
                         "to this JSON file, for matching them with profiler records")
    ap.add_argument("--profile-ops", default="ffn_up",
                    help="operations timed with HIP events during the timed steps: any of "
                         "ffn_up,ffn_down,h2d,combine,route_topk,permute,score_retain,"
                         "layer_adapt ('' for none)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU: the expert-offloading layer path runs on a single "
              "GPU and has no multi-GPU mode (run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2609_33385_amd import oled
    from paper_2609_33385_amd import workload as W

    w = W.WORKLOADS[args.workload]
    if args.capacity is not None:
        w = w.replace(capacity=args.capacity)
    L, T, E = w.n_layers, w.tokens, w.n_experts
    torch.cuda.set_device(0)
    lib = oled.load()

    t0 = time.time()
    n_blocks = args.pool_blocks or min(L * E, (16 << 30) // w.expert_bytes)
    pool = oled.PinnedPool(n_blocks, w.expert_bytes)
    fill_pool_device(pool, w, args.seed)
    n_total = args.warmup + max(args.steps, args.phase_steps)
    logits, xs, conf = make_inputs(w, args.seed, n_total)
    y = torch.empty((T, w.hidden), dtype=torch.bfloat16, device="cuda")
    prof = oled.profile_mask(*[o for o in args.profile_ops.split(",") if o])
    coop = None
    if args.coop:
        coop = profile_coop(w, pool, logits, xs, conf, args)
        log(f"coop split constants: {coop}")
    def make_ctx(profile_ops):
        return oled.Context(w.hidden, w.inter, E, w.top_k, L, w.capacity, T, w.dtype, pool.ptr,
                            pool.n_blocks, W.host_block_of(w, pool.n_blocks),
                            profile_ops=profile_ops, copy_mode=args.copy_mode,
                            adapt_period=args.adapt_period, coop=coop)
    ctx = make_ctx(prof)
    log(f"setup {time.time() - t0:.1f}s: pool {pool.n_blocks} x {w.expert_bytes >> 20} MiB pinned")

    s = torch.cuda.current_stream()
    sp = s.cuda_stream
    lg_p = [[logits[g, l].data_ptr() for l in range(L)] for g in range(n_total)]
    x_p = [[xs[g, l].data_ptr() for l in range(L)] for g in range(n_total)]
    c_p = [conf[g].data_ptr() for g in range(n_total)]
    y_p = y.data_ptr()

    def step_on(c, g):
        h = c.ctx
        for l in range(L):
            if lib.route_block(h, l, lg_p[g][l], T, sp):
                raise oled.OledError(1, oled.last_error(h))
            if lib.moe_forward_cached(h, l, x_p[g][l], y_p, sp):
                raise oled.OledError(1, oled.last_error(h))
            if coop:
                if lib.apply_misses_coop(h, l, c_p[g], None):
                    raise oled.OledError(1, oled.last_error(h))
            elif lib.apply_misses(h, l, None, None):
                raise oled.OledError(1, oled.last_error(h))
            if lib.score_and_retain(h, l, c_p[g], sp):
                raise oled.OledError(1, oled.last_error(h))

    def step(g):
        step_on(ctx, g)

    for g in range(args.warmup):
        step(g)
    torch.cuda.synchronize()
    if args.calibration:
        ca = torch.ones(64 << 20, dtype=torch.float32, device="cuda")
        cb = torch.empty_like(ca)
        for _ in range(2):
            torch.neg(ca, out=cb)
        torch.cuda.synchronize()
        del ca, cb
    ctx.profile_collect()            # drop warm-up timings and counts
    ctx.collect_stats()
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for g in range(args.warmup, n_total):
        step(g)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start
    ops = ctx.profile_collect()
    st = ctx.collect_stats()
    stats = {"hits": st["n_hits"], "misses": st["n_misses"], "active": st["n_active"],
             "h2d_bytes": st["h2d_bytes"], "layer_iters": st["layer_iters"],
             "cpu": st["n_cpu_executed"]}

    def agg(name, transfer=None):
        """Launches of one kind; transfer True/False: only those that did / did
        not also move miss weights host->device."""
        sel = [o for o in ops if o[0] == name and
               (transfer is None or (o[5] > 0) == transfer)]
        ms = sum(o[2] for o in sel)
        return dict(n=len(sel), ms=ms, bytes=sum(o[3] for o in sel), flops=sum(o[4] for o in sel),
                    h2d=sum(max(0, o[5]) for o in sel))

    # the gate/up GEMM's HBM roofline over the launches that moved no miss
    # weights (a launch that also transfers misses runs as long as its PCIe reads)
    up, down = agg("ffn_up", transfer=False), agg("ffn_down", transfer=False)
    up_x, down_x, h2d = agg("ffn_up", transfer=True), agg("ffn_down", transfer=True), agg("h2d")
    adapt = agg("layer_adapt")
    up_gbs = (up["bytes"] / 1e9) / (up["ms"] / 1e3) if up["ms"] > 0 else 0.0
    ffn_ms = up["ms"] + down["ms"]
    ffn_tflops = ((up["flops"] + down["flops"]) / 1e12) / (ffn_ms / 1e3) if ffn_ms > 0 else 0.0
    ffn_gbs = ((up["bytes"] + down["bytes"]) / 1e9) / (ffn_ms / 1e3) if ffn_ms > 0 else 0.0
    # host-to-device rate of the miss transfers: inside the gate/up and down
    # launches that carried them (shader), or the copy-engine copies (sdma)
    x_ms = up_x["ms"] + down_x["ms"] + h2d["ms"]
    x_bytes = up_x["h2d"] + down_x["h2d"] + h2d["h2d"]
    h2d_rate = round((x_bytes / 1e9) / (x_ms / 1e3), 2) if x_ms > 0 else None
    if args.launch_log:
        with open(args.launch_log, "w") as f:
            json.dump({"ffn_up": [[o[3], o[5]] for o in ops if o[0] == "ffn_up"]}, f)
    value = args.steps * L * T / elapsed
    li = max(1, stats["layer_iters"])
    out = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "layer-tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(elapsed / args.steps * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded router logits, activations, confidence; random-init bf16 experts)",
        "config": {"workload": (f"LLaDA-MoE-like layer stack, bf16: hidden {w.hidden}, {E} experts, "
                                f"top-{w.top_k}, expert intermediate {w.inter}, {L} MoE layers, "
                                f"batch {w.batch} x block {w.block} tokens, {w.n_iters} denoising "
                                f"iterations per block, expert cache {w.capacity}/{E} "
                                f"({round(100 * w.capacity / E)}%) per layer"
                                + (f", router logits with Zipf({w.zipf_s}) expert popularity"
                                   if w.zipf_s else "")
                                + (f", iteration noise N(0, {w.sigma_it})"
                                   if w.sigma_it != 0.3 else "")
                                + (", cooperative CPU compensation" if coop else "")
                                + (f", layer-adaptive sizing every {args.adapt_period} iterations"
                                   if args.adapt_period else "")),
                   "hidden": w.hidden, "n_experts": E, "top_k": w.top_k, "inter": w.inter,
                   "n_layers": L, "tokens_per_iteration": T, "iterations_per_block": w.n_iters,
                   "capacity": w.capacity, "host_pool_blocks": n_blocks},
        "roofline": {"kernel": "grouped gate/up SwiGLU GEMM (k_ffn up), launches that moved no "
                               "miss weights", "bound": "hbm",
                     "achieved": round(up_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(up_gbs / HBM_PEAK_GBS, 4), "traffic": measured_traffic(),
                     "launches": up["n"], "avg_launch_us": round(up["ms"] / max(1, up["n"]) * 1e3, 2),
                     "bytes_per_launch": int(up["bytes"] / max(1, up["n"]))},
        "detail": {
            "ffn_up_down_GBps": round(ffn_gbs, 1) if down["n"] else None,
            "ffn_up_mfma_util": round((up["flops"] / 1e12) / (up["ms"] / 1e3) / MFMA_BF16_PEAK_TFLOPS, 5)
                                if up["ms"] > 0 else None,
            "ffn_mfma_util": round(ffn_tflops / MFMA_BF16_PEAK_TFLOPS, 5) if down["n"] else None,
            "ffn_ms_per_step": round(ffn_ms / args.steps, 4) if down["n"] else None,
            "copy_mode": args.copy_mode,
            "adapt_period": args.adapt_period,
            "layer_adapt_us": round(adapt["ms"] / adapt["n"] * 1e3, 2) if adapt["n"] else None,
            "h2d_GBps": h2d_rate,
            "transfer_launches": up_x["n"] + down_x["n"] + h2d["n"],
            "profiled_ops": args.profile_ops,
            "hits_per_layer_iter": round(stats["hits"] / li, 3),
            "misses_per_layer_iter": round(stats["misses"] / li, 3),
            "active_per_layer_iter": round(stats["active"] / li, 3),
            "cache_util": round(stats["hits"] / li / max(1, w.capacity), 4),
            "h2d_MiB_per_step": round(stats["h2d_bytes"] / args.steps / 2 ** 20, 2),
            "coop": coop,
            "cpu_executed_per_layer_iter": round(stats["cpu"] / li, 3) if coop else None,
        },
    }
    ctx.close()
    if args.phase_steps > 0:
        out["detail"]["phase_pass"] = phase_pass(w, pool, step_on, make_ctx, args)
    pool.free()
    if not args.no_cpu_baseline and args.workload <= 3:
        # (the E=128 stacks' float64 oracle takes minutes per layer-iteration)
        out["cpu_baseline"] = cpu_baseline(w, args.seed)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
