"""Block-MoE layer throughput on one MI355X under partial expert residency.

Headline workload (default, --workload 4): the E=128 layer stack in bf16 -
hidden 4096, 128 experts, top-8, expert SwiGLU intermediate 1536, 48 MoE
layers, batch 16 x block 64 = 1024 tokens per iteration, 16 denoising
iterations per block, router logits with a Zipf(1.1) expert popularity, expert
cache 51 of 128 experts per layer (40%). One step is one denoising iteration
through all 48 layers: per layer route_block -> moe_forward_cached (the cached
experts' GEMMs; their first workgroups copy the misses' gate/up weights from
pinned host memory over PCIe) -> apply_misses (the cached experts' down GEMM
with the copy of the misses' down weights, then the misses' GEMMs) ->
score_and_retain (combine, priorities, retention). With --copy-mode sdma the
misses are copied by hipMemcpyAsync on a copy stream instead. Blocks follow
each other without resetting the caches; the warm-up steps cover the cold
start.

Inputs are generated before timing and resident in HBM: router logits and
confidence by the seeded numpy generators of workload.py, activations by
torch's seeded Philox generator on the GPU (N(0, 0.02^2) in bf16; the routing
does not depend on them). Expert weights (N(0, 0.02^2), drawn on the GPU)
live in a pinned host pool and reach the GPU only through cache misses; the
E=128 stacks alias their 6144 experts onto 448 host blocks (16 GiB), which
changes neither the bytes per miss nor the routing.

Prints one JSON line: the layer-token throughput of the timed steps, the
roofline of the dominant kernel (the gate/up GEMM launch, HIP events on its
dispatches during the timed steps: HBM fraction over all launches, over the
launches without a transfer, and the transfer launches against the host
link), the host link over the whole step, and the CPU oracle timed on a
bounded sample (single-threaded and on all cores). Under `detail`, outside the
timed region: a per-phase pass on a second context, the same stack with every
expert cached (capacity E), and the 64-expert stack with 32 tokens per
iteration as a secondary line.
"""
from __future__ import annotations

import argparse
import concurrent.futures
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0            # MI355X HBM3E
MFMA_BF16_PEAK_TFLOPS = 2500.0   # dense bf16 MFMA
PCIE_GEN5_X16_GBS = 63.0         # 32 GT/s x 16 lanes, 128b/130b, one direction
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
    chunk = max(1, min(chunk, (1 << 30) // (per * 4)))
    for b0 in range(0, pool.n_blocks, chunk):
        n = min(chunk, pool.n_blocks - b0)
        v = (torch.randn(n * per, generator=g, device="cuda") * 0.02).to(torch.bfloat16)
        host[b0 * per:(b0 + n) * per].copy_(v.view(torch.int16))
    torch.cuda.synchronize()


def make_inputs(w, seed: int, n_steps: int):
    """Device tensors: logits[g][l] [T][E] fp32, x[g][l] [T][H] dtype, conf[g] [T].

    Logits and confidence come from workload.py (numpy, drawn on a thread
    pool); activations from torch's Philox generator on the GPU."""
    import torch
    from paper_2609_33385_amd import workload as W
    N, L = w.n_iters, w.n_layers
    n_blocks = (n_steps + N - 1) // N
    lg = np.empty((n_blocks * N, L, w.tokens, w.n_experts), np.float32)

    def one(bl):
        b, l = bl
        lg[b * N:(b + 1) * N, l] = W.logits_block(w, seed, l, b)

    with concurrent.futures.ThreadPoolExecutor(16) as ex:
        list(ex.map(one, [(b, l) for b in range(n_blocks) for l in range(L)]))
    cf = np.stack([W.confidence(w, seed, g // N, g % N) for g in range(n_steps)])
    dt = torch.float32 if w.dtype == "f32" else torch.bfloat16
    gen = torch.Generator(device="cuda")
    gen.manual_seed(seed + 7919)
    xs = torch.empty((n_steps, L, w.tokens, w.hidden), dtype=dt, device="cuda")
    for g in range(n_steps):
        xs[g].copy_(torch.randn((L, w.tokens, w.hidden), generator=gen, device="cuda") * 0.02)
    return torch.from_numpy(lg[:n_steps]).cuda(), xs, torch.from_numpy(cf).cuda()


FFN_SOURCE = os.path.join(ROOT, "paper_2609_33385_amd", "csrc", "ffn.hip")


def traffic_file(wid: int) -> str:
    name = {2: "llada40", 4: "e128_zipf40"}.get(wid, f"workload{wid}")
    return os.path.join(ROOT, "profiles", f"k_ffn_up_{name}_traffic.json")


def measured_traffic(wid: int):
    """HBM bytes per gate/up GEMM launch from the committed counter summary of
    this workload, or None if there is none or the kernel source changed since
    the counters were taken."""
    import hashlib
    try:
        with open(traffic_file(wid)) as f:
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
    t_h2d = w.expert_bytes / (pinned_h2d_gbps(pool, w) * 1e3)   # microseconds
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


def pinned_h2d_gbps(pool, w, n: int = 40):
    """Host-to-device rate of plain copies of one expert block from the pinned
    pool (hipMemcpyAsync, n copies after 4 untimed ones). Taken after the
    timed steps: on a link that has been idle the first copies run slower."""
    import torch
    host = torch.from_numpy(pool.view(np.uint8)[: w.expert_bytes])
    dev = torch.empty(w.expert_bytes, dtype=torch.uint8, device="cuda")
    for _ in range(4):
        dev.copy_(host, non_blocking=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(n):
        dev.copy_(host, non_blocking=True)
    torch.cuda.synchronize()
    return n * w.expert_bytes / (time.perf_counter() - t0) / 1e9


def agg(ops, name, transfer=None):
    """Launches of one kind; transfer True/False: only those that did / did
    not also move miss weights host->device."""
    sel = [o for o in ops if o[0] == name and (transfer is None or (o[5] > 0) == transfer)]
    ms = sum(o[2] for o in sel)
    return dict(n=len(sel), ms=ms, bytes=sum(o[3] for o in sel), flops=sum(o[4] for o in sel),
                h2d=sum(max(0, o[5]) for o in sel))


def rate(a):
    """GB/s of a launch group's algorithmic bytes, and its HBM fraction."""
    if a["n"] == 0 or a["ms"] <= 0:
        return None, None
    gbs = (a["bytes"] / 1e9) / (a["ms"] / 1e3)
    return round(gbs, 1), round(gbs / HBM_PEAK_GBS, 4)


def phase_pass(w, pool, step_fn, make_ctx, args, link):
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
        a = agg(ops, name)
        if not a["n"]:
            continue
        gbs, frac = rate(a)
        phases[name] = {"launches": a["n"], "us_per_layer_iter": round(a["ms"] * 1e3 / n_li, 2),
                        "avg_us": round(a["ms"] * 1e3 / a["n"], 2), "GBps": gbs, "hbm_frac": frac}
        calm = agg(ops, name, transfer=False)
        if name != "h2d" and 0 < calm["n"] < a["n"]:
            # launches that also carried miss weights run as long as the PCIe reads
            cgb, cfr = rate(calm)
            phases[name]["without_transfer"] = {
                "launches": calm["n"], "avg_us": round(calm["ms"] * 1e3 / calm["n"], 2),
                "GBps": cgb, "hbm_frac": cfr}
    # launches on the compute stream (copy-engine copies run beside them)
    t_layer = [sum(o[2] for o in gr if o[0] != "h2d") for gr in groups]
    xfer = [sum(max(0, o[5]) for o in gr) for gr in groups]
    calm_t = [t for t, b in zip(t_layer, xfer) if b == 0]
    t_comp = float(np.mean(calm_t)) if calm_t else None
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
            "overlap_efficiency": overlap}


def cpu_info():
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    model = ln.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        usable = len(os.sched_getaffinity(0))
    except AttributeError:
        usable = os.cpu_count()
    return model, os.cpu_count(), usable


def cpu_baseline(w, seed: int, pool_blocks: int, experts_per_point: int = 48):
    """The oracle on the host's cores, on a bounded sample of the workload.

    Control path (routing, permutation, hit/miss sets, priorities, retention:
    O1-O3, O6-O8) on every iteration of block 0 of layers {0, L/2, L-1}, timed
    on iterations {0, 1, N-1} of each (9 layer-iterations). Expert FFN and
    combine (O4-O5) on 3 of those layer-iterations, for `experts_per_point`
    active experts each, spread over the experts sorted by routed rows (the
    oracle's output restricted to their routes). Extrapolation per
    layer-iteration: s = mean control time + mean |A| x mean time per sampled
    expert, and layer-tokens/s = T / s. Timed twice: BLAS on every thread
    numpy has, and on one thread (threadpoolctl). Weights: numpy draws of the
    same host blocks (aliasing as the GPU pool), outside the timing."""
    from threadpoolctl import threadpool_info, threadpool_limits

    from oracle import oled_oracle as O
    from paper_2609_33385_amd import workload as W
    L, N, E, T = w.n_layers, w.n_iters, w.n_experts, w.tokens
    layers = sorted({0, L // 2, L - 1})
    iters = sorted({0, min(1, N - 1), N - 1})
    ffn_at = {(layers[0], iters[min(1, len(iters) - 1)]), (layers[len(layers) // 2], N - 1),
              (layers[-1], iters[min(1, len(iters) - 1)])}
    hbo = W.host_block_of(w, pool_blocks)
    t_ctrl, samples = [], []
    for l in layers:
        lgb = W.logits_block(w, seed, l, 0)
        res = np.zeros(E, bool)
        for i in range(N):
            conf = W.confidence(w, seed, 0, i)
            t0 = time.perf_counter()
            st = O.layer_step(lgb[i], conf, res, w.top_k, w.capacity)
            dt = time.perf_counter() - t0
            res = st["resident_after"]
            if i in iters:
                t_ctrl.append(dt)
            if (l, i) in ffn_at:
                act = [e for e in np.argsort(st["counts"], kind="stable") if st["counts"][e] > 0]
                m = min(experts_per_point, len(act))
                pick = [int(act[int((j + 0.5) * len(act) / m)]) for j in range(m)]
                samples.append(dict(l=l, i=i, st=st, n_active=len(act), experts=pick,
                                    x=O.decode(W.activations(w, seed, l, 0, i))))
    blocks = {int(hbo[s["l"] * E + e]) for s in samples for e in s["experts"]}
    raw = W.expert_blocks(w, seed, sorted(blocks))       # drawn outside the timing

    def ffn_times():
        out = []
        for s in samples:
            def weights(e, l=s["l"]):
                return W.split_expert(w, O.decode(raw[int(hbo[l * E + e])]))
            for e in s["experts"]:
                t0 = time.perf_counter()
                O.moe_output(s["x"], s["st"]["idx"], s["st"]["gates"], weights, experts=[e])
                out.append(time.perf_counter() - t0)
        return out

    threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    t_all = ffn_times()
    with threadpool_limits(1):
        t_one = ffn_times()
    a_mean = float(np.mean([s["n_active"] for s in samples]))
    c_mean = float(np.mean(t_ctrl))
    s_all = c_mean + a_mean * float(np.mean(t_all))
    s_one = c_mean + a_mean * float(np.mean(t_one))
    model, ncpu, usable = cpu_info()
    formula = (f"s per layer-iteration = mean control {c_mean:.4f} s + mean |A| {a_mean:.1f} x "
               f"mean s per sampled expert ({np.mean(t_all):.4f} s on {threads} BLAS threads, "
               f"{np.mean(t_one):.4f} s on one); layer-tokens/s = {T} / s")
    return {"value": round(T / s_all, 2), "unit": "layer-tokens/s", "cores": int(threads),
            "kind": "oracle",
            "sample": (f"control path on {len(t_ctrl)} layer-iterations (layers {layers} x "
                       f"iterations {iters} of block 0), expert FFN + combine for "
                       f"{len(t_all)} experts on {len(samples)} of them; "
                       f"{sum(t_ctrl) + sum(t_all) + sum(t_one):.1f} s of CPU work; {formula}"),
            "single_thread": {"value": round(T / s_one, 2), "cores": 1},
            "cpu_model": model, "nproc": ncpu, "usable_cpus": usable}


def timed_window(ctx, step_fn, warmup: int, steps: int, calibration: bool = False):
    """Warm-up, then exactly `steps` timed steps between two device syncs."""
    import torch
    for g in range(warmup):
        step_fn(ctx, g)
    torch.cuda.synchronize()
    if calibration:
        ca = torch.ones(64 << 20, dtype=torch.float32, device="cuda")
        cb = torch.empty_like(ca)
        for _ in range(2):
            torch.neg(ca, out=cb)
        torch.cuda.synchronize()
        del ca, cb
    ctx.profile_collect()            # drop warm-up timings and counts
    ctx.collect_stats()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for g in range(warmup, warmup + steps):
        step_fn(ctx, g)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    return elapsed, ctx.profile_collect(), ctx.collect_stats()


def make_stepper(lib, oled, w, logits, xs, conf, coop):
    """step_on(ctx, g): step g through every layer with the ABI calls."""
    import torch
    L, T = w.n_layers, w.tokens
    n = logits.shape[0]
    sp = torch.cuda.current_stream().cuda_stream
    lg_p = [[logits[g, l].data_ptr() for l in range(L)] for g in range(n)]
    x_p = [[xs[g, l].data_ptr() for l in range(L)] for g in range(n)]
    c_p = [conf[g].data_ptr() for g in range(n)]
    y = torch.empty((T, w.hidden), dtype=xs.dtype, device="cuda")
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

    step_on.keep = y
    return step_on


def workload_text(w, coop=None, adapt=0):
    return (f"block-MoE layer stack, bf16: hidden {w.hidden}, {w.n_experts} experts, "
            f"top-{w.top_k}, expert intermediate {w.inter}, {w.n_layers} MoE layers, "
            f"batch {w.batch} x block {w.block} tokens, {w.n_iters} denoising iterations per "
            f"block, expert cache {w.capacity}/{w.n_experts} "
            f"({round(100 * w.capacity / w.n_experts)}%) per layer"
            + (f", router logits with Zipf({w.zipf_s}) expert popularity" if w.zipf_s else "")
            + (f", iteration noise N(0, {w.sigma_it})" if w.sigma_it != 0.3 else "")
            + (", cooperative CPU compensation" if coop else "")
            + (f", layer-adaptive sizing every {adapt} iterations" if adapt else ""))


def roofline_object(ops, wid, link):
    """The dominant kernel (gate/up GEMM launches) against HBM over every timed
    launch; the launches without a transfer alone; the transfer launches
    against the host link."""
    up_all = agg(ops, "ffn_up")
    calm = agg(ops, "ffn_up", transfer=False)
    xf = agg(ops, "ffn_up", transfer=True)
    gbs, frac = rate(up_all)
    obj = {"kernel": "k_ffn<up>: grouped gate/up SwiGLU GEMM of the cached experts (its first 64 "
                     "workgroups also copy the misses' gate/up weights host->device), every "
                     "timed launch",
           "bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": frac,
           "traffic": measured_traffic(wid), "launches": up_all["n"],
           "avg_launch_us": round(up_all["ms"] / max(1, up_all["n"]) * 1e3, 2),
           "bytes_per_launch": int(up_all["bytes"] / max(1, up_all["n"]))}
    cg, cf = rate(calm)
    obj["without_transfer"] = ({"launches": calm["n"], "achieved": cg, "frac": cf,
                                "avg_launch_us": round(calm["ms"] / calm["n"] * 1e3, 2)}
                               if calm["n"] else None)
    if xf["n"]:
        h2d = (xf["h2d"] / 1e9) / (xf["ms"] / 1e3)
        xg, xfr = rate(xf)
        obj["transfer_launches"] = {
            "launches": xf["n"], "avg_launch_us": round(xf["ms"] / xf["n"] * 1e3, 2),
            "h2d_bytes_per_launch": int(xf["h2d"] / xf["n"]), "h2d_GBps": round(h2d, 2),
            "pinned_copy_GBps": round(link, 2), "frac_of_pinned_copy": round(h2d / link, 4),
            "pcie_gen5_x16_GBps": PCIE_GEN5_X16_GBS,
            "frac_of_pcie_gen5_x16": round(h2d / PCIE_GEN5_X16_GBS, 4),
            "hbm_GBps": xg, "hbm_frac": xfr}
    else:
        obj["transfer_launches"] = None
    return obj


def full_residency(w, pool, step_on, make_ctx_cap, steps: int):
    """The same stack with every expert cached (capacity E): the steps to be
    timed run once untimed (fetching every expert they activate; at capacity
    E nothing is evicted), then the same `steps` steps are timed with the GEMM
    launches timed. No transfers in the timed steps: the layer's HBM-bound
    cost."""
    from paper_2609_33385_amd import oled
    ctx = make_ctx_cap(w.n_experts, oled.profile_mask("ffn_up", "ffn_down", "ffn_dense_up",
                                                      "ffn_dense_down", "combine", "route_topk",
                                                      "permute"))
    try:
        for g in range(steps):
            step_on(ctx, g)
        elapsed, ops, st = timed_window(ctx, step_on, 0, steps)
    finally:
        ctx.close()
    L, T = w.n_layers, w.tokens
    li = max(1, st["layer_iters"])
    kern = {}
    for name in ("route_topk", "permute", "ffn_up", "ffn_down", "ffn_dense_up", "ffn_dense_down",
                 "combine"):
        a = agg(ops, name)
        if a["n"]:
            g, f = rate(a)
            kern[name] = {"launches": a["n"], "avg_us": round(a["ms"] / a["n"] * 1e3, 2),
                          "GBps": g, "hbm_frac": f}
    gemm = [agg(ops, n) for n in ("ffn_up", "ffn_down", "ffn_dense_up", "ffn_dense_down")]
    g_ms = sum(a["ms"] for a in gemm)
    g_by = sum(a["bytes"] for a in gemm)
    g_fl = sum(a["flops"] for a in gemm)
    return {"capacity": w.n_experts, "steps": steps,
            "value": round(steps * L * T / elapsed, 1),
            "ms_per_step": round(elapsed / steps * 1e3, 3),
            "misses_per_layer_iter": round(st["n_misses"] / li, 3),
            "active_per_layer_iter": round(st["n_active"] / li, 3),
            "gemm_hbm_frac": round((g_by / 1e9) / (g_ms / 1e3) / HBM_PEAK_GBS, 4) if g_ms else None,
            "gemm_mfma_util": round((g_fl / 1e12) / (g_ms / 1e3) / MFMA_BF16_PEAK_TFLOPS, 4)
            if g_ms else None,
            "gemm_ms_per_layer_iter": round(g_ms / li, 4),
            "kernels": kern}


def run_workload(w, args, lib, oled, coop=None, headline=True):
    """Pool, inputs, the timed window (optionally repeated, the cache reset
    before each), and the figures of the line. Returns (record, context
    factory, stepper, pool, link rate)."""
    import torch
    from paper_2609_33385_amd import workload as W
    L, T, E = w.n_layers, w.tokens, w.n_experts
    t0 = time.time()
    n_blocks = args.pool_blocks or min(L * E, (16 << 30) // w.expert_bytes)
    pool = oled.PinnedPool(n_blocks, w.expert_bytes)
    fill_pool_device(pool, w, args.seed)
    warmup, steps = (args.warmup, args.steps) if headline else (8, 64)
    phase_steps = args.phase_steps if args.phase_steps >= 0 else (4 if E > 64 else 8)
    n_total = warmup + max(steps, phase_steps if headline else 0)
    if headline:
        n_total = max(n_total, 2 + args.full_steps)
    logits, xs, conf = make_inputs(w, args.seed, n_total)
    log(f"setup {time.time() - t0:.1f}s: {w.name}, pool {pool.n_blocks} x "
        f"{w.expert_bytes >> 20} MiB pinned, inputs for {n_total} steps")
    if coop is not None and not isinstance(coop, dict):
        coop = profile_coop(w, pool, logits, xs, conf, args)
        log(f"coop split constants: {coop}")
    step_on = make_stepper(lib, oled, w, logits, xs, conf, coop)
    prof = oled.profile_mask(*[o for o in args.profile_ops.split(",") if o])

    def make_ctx(profile_ops, capacity=None):
        return oled.Context(w.hidden, w.inter, E, w.top_k, L,
                            w.capacity if capacity is None else capacity, T, w.dtype, pool.ptr,
                            pool.n_blocks, W.host_block_of(w, pool.n_blocks),
                            profile_ops=profile_ops, copy_mode=args.copy_mode,
                            adapt_period=args.adapt_period, coop=coop)

    ctx = make_ctx(prof)
    runs = []
    try:
        for r in range(args.repeats if headline else 1):
            if r:
                ctx.reset_cache()
            elapsed, ops, st = timed_window(ctx, step_on, warmup, steps,
                                            calibration=args.calibration and headline)
            runs.append((elapsed, ops, st))
            log(f"{w.name} run {r}: {steps * L * T / elapsed:.1f} layer-tokens/s, "
                f"{elapsed / steps * 1e3:.2f} ms per step")
    finally:
        ctx.close()
    link = pinned_h2d_gbps(pool, w)
    log(f"pinned host-to-device copies: {link:.1f} GB/s")
    elapsed = float(np.mean([r[0] for r in runs]))
    ops = [o for r in runs for o in r[1]]
    st = {k: sum(r[2][k] for r in runs) for k in runs[0][2]}
    if args.launch_log and headline:
        os.makedirs(os.path.dirname(os.path.abspath(args.launch_log)), exist_ok=True)
        with open(args.launch_log, "w") as f:   # every timed profiled operation, in order
            json.dump({"ops": [[o[0], o[1], o[2], o[3], o[4], o[5]] for o in runs[-1][1]]}, f)
    li = max(1, st["layer_iters"])
    ms_step = elapsed / steps * 1e3
    h2d_step = st["h2d_bytes"] / (steps * len(runs))
    link_step = (h2d_step / 1e9) / (ms_step / 1e3)
    up = agg(ops, "ffn_up")
    rec = {
        "value": round(steps * L * T / elapsed, 1),
        "ms_per_step": round(ms_step, 4),
        "steps": steps, "warmup": warmup,
        "runs": [round(steps * L * T / r[0], 1) for r in runs],
        "config": {"workload": workload_text(w, coop, args.adapt_period), "hidden": w.hidden,
                   "n_experts": E, "top_k": w.top_k, "inter": w.inter, "n_layers": L,
                   "tokens_per_iteration": T, "iterations_per_block": w.n_iters,
                   "capacity": w.capacity, "host_pool_blocks": n_blocks},
        "roofline": roofline_object(ops, w.wid, link),
        "host_link_per_step": {"h2d_MiB_per_step": round(h2d_step / 2 ** 20, 2),
                               "GBps": round(link_step, 2),
                               "frac_of_pinned_copy": round(link_step / link, 4),
                               "frac_of_pcie_gen5_x16": round(link_step / PCIE_GEN5_X16_GBS, 4),
                               "pinned_copy_GBps": round(link, 2)},
        "ffn_up_mfma_util": round((up["flops"] / 1e12) / (up["ms"] / 1e3) / MFMA_BF16_PEAK_TFLOPS, 5)
        if up["ms"] > 0 else None,
        "copy_mode": args.copy_mode,
        "hits_per_layer_iter": round(st["n_hits"] / li, 3),
        "misses_per_layer_iter": round(st["n_misses"] / li, 3),
        "active_per_layer_iter": round(st["n_active"] / li, 3),
        "cache_util": round(st["n_hits"] / li / max(1, w.capacity), 4),
        "coop": coop if isinstance(coop, dict) else None,
        "cpu_executed_per_layer_iter": round(st["n_cpu_executed"] / li, 3) if coop else None,
    }
    if headline and phase_steps > 0:
        args.phase_steps = phase_steps
        rec["phase_pass"] = phase_pass(w, pool, step_on, lambda p: make_ctx(p), args, link)
    if headline and args.full_steps > 0 and args.adapt_period == 0 and coop is None:
        try:
            rec["full_residency"] = full_residency(w, pool, step_on,
                                                   lambda cap, p: make_ctx(p, capacity=cap),
                                                   args.full_steps)
        except oled.OledError as e:     # the slot pool of every expert may not fit
            rec["full_residency"] = {"capacity": w.n_experts, "error": str(e)}
        log(f"full residency: {rec['full_residency'].get('value')} layer-tokens/s")
    del logits, xs, conf
    pool.free()
    torch.cuda.empty_cache()
    return rec


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--capacity", type=int, default=None, help="experts cached per layer")
    ap.add_argument("--workload", type=int, default=4, choices=[2, 3, 4, 5],
                    help="4: the E=128 stack (hidden 4096, 48 layers, 1024 tokens, Zipf "
                         "popularity, 40%%; the headline); 5: its stress form (20%%, iteration "
                         "noise 1.5); 2: the 64-expert stack with 32 tokens per iteration (40%%); "
                         "3: the same with batch 8 x block 32 = 256 tokens")
    ap.add_argument("--repeats", type=int, default=1,
                    help="timed windows, each after a cache reset and the warm-up; the value is "
                         "their mean (the paper's protocol takes 3)")
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
    ap.add_argument("--no-secondary", action="store_true",
                    help="skip the 64-expert, 32-token stack measured after the headline")
    ap.add_argument("--full-steps", type=int, default=8,
                    help="timed steps of the same stack with every expert cached (0: skip)")
    ap.add_argument("--phase-steps", type=int, default=-1,
                    help="after the timed steps, this many steps on a second context with every "
                         "operation timed: per-phase times and overlap efficiency (0: skip; "
                         "default 4 on the E=128 stacks, 8 otherwise)")
    ap.add_argument("--calibration", action="store_true",
                    help="between warm-up and timed steps, run a plain streaming kernel of known "
                         "traffic (torch negation over 256 MiB fp32: 256 MiB read, 256 MiB "
                         "written) to scale hardware byte counters")
    ap.add_argument("--copy-mode", default="shader", choices=["shader", "sdma"],
                    help="transfer of the misses: workgroups of the hit GEMM launches (shader) "
                         "or hipMemcpyAsync on a copy stream (sdma)")
    ap.add_argument("--launch-log", default=None,
                    help="write the timed profiled operations in order ([op, layer, ms, bytes, "
                         "flops, h2d bytes] each) to this JSON file, for matching them with "
                         "profiler records")
    ap.add_argument("--profile-ops", default="ffn_up",
                    help="operations timed with HIP events during the timed steps: any of "
                         "ffn_up,ffn_down,h2d,combine,route_topk,permute,score_retain,"
                         "layer_adapt ('' for none)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU and has no multi-GPU mode: run it with --gpus 1",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2609_33385_amd import oled
    from paper_2609_33385_amd import workload as W

    w = W.WORKLOADS[args.workload]
    if args.capacity is not None:
        w = w.replace(capacity=args.capacity)
    torch.cuda.set_device(0)
    lib = oled.load()
    rec = run_workload(w, args, lib, oled, coop=True if args.coop else None)
    out = {
        "metric": METRIC,
        "value": rec.pop("value"),
        "unit": "layer-tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": rec.pop("ms_per_step"),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded router logits, activations, confidence; random-init bf16 "
                "experts)",
        "config": rec.pop("config"),
        "roofline": rec.pop("roofline"),
        "detail": rec,
    }
    for k in ("steps", "warmup"):
        rec.pop(k)
    if not args.no_secondary and args.workload != 2:
        w2 = W.WORKLOADS[2]
        sec = run_workload(w2, args, lib, oled, headline=False)
        out["detail"]["secondary"] = {
            "workload": sec["config"]["workload"], "value": sec["value"],
            "ms_per_step": sec["ms_per_step"], "steps": sec["steps"], "warmup": sec["warmup"],
            "misses_per_layer_iter": sec["misses_per_layer_iter"],
            "host_link_per_step": sec["host_link_per_step"], "roofline": sec["roofline"]}
    if not args.no_cpu_baseline:
        t0 = time.time()
        out["cpu_baseline"] = cpu_baseline(w, args.seed, out["config"]["host_pool_blocks"])
        log(f"cpu baseline {time.time() - t0:.1f}s")
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
