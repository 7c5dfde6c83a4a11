"""Supplementary measurements on one MI355X, beside the headline bench.

--gemm: the prefill-like shape on which the grouped SwiGLU GEMM is compute
  bound: LLaDA-MoE-like dims of the 48-layer stack (hidden 4096, 128
  experts, top-8, expert intermediate 1536, bf16; router logits without
  expert popularity bias) with 16384 tokens (256 sequences x 64), so about
  1024 routed rows per expert. One layer with
  every expert cached (C = E): iteration 0 fills the cache, iterations 1..N
  are timed. Every expert with 128+ rows runs as dense tiles; the line
  reports their MFMA utilisation against 2.5 PFLOP/s dense bf16 (device time
  between HIP events on the compute stream around each launch) and checks
  sampled output rows against the oracle.

--route: the routing kernels on a batched input of 1 GiB: top-k and gates
  over the fp32 router logits of 32 layers x 65535 tokens x 128 experts,
  then the histogram / scan / permutation and the retention of each layer's
  524280 routes; per-launch device times (HIP events) and HBM fractions of
  the algorithmic bytes against 8 TB/s; for context, the read rate of
  torch.amax over each token's experts and of torch.sum on the same 1 GiB.

--vendor: context for --gemm: the vendor library's batched bf16 GEMM
  (torch.bmm, which calls hipBLASLt) on plain contiguous operands of the
  same dimensions: 128 experts x 1024 rows against the gate/up weights
  (4096 -> 3072) and the down weights (1536 -> 4096), bf16 output, event
  timed; then the down product right behind the gate/up product, as a layer
  runs them. It does none of the routed gather, SwiGLU or expert-sorted rows.

--gate: the gate GEMM of route_block_gate (logits = x W_gate^T, fp32
  accumulation) on the 40% stack's shape (32 tokens, hidden 2048, 64 experts),
  its batch-8 form (256 tokens), the E=128 stack (1024 tokens, hidden 4096)
  and the prefill-like block (16384 tokens, hidden 4096, 128 experts):
  device time per launch (HIP events), TFLOP/s and the HBM fraction of its
  algorithmic bytes (x, W_gate, logits).

Each mode prints one JSON line. Inputs are seeded and synthetic.
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

HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def gemm(args):
    import torch
    from oracle import oled_oracle as O
    from paper_2609_33385_amd import harness as HN
    from paper_2609_33385_amd import oled
    from paper_2609_33385_amd import workload as W

    w = W.WORKLOADS[5].replace(wid=400, name="prefill", batch=256, block=64, n_layers=1,
                               n_iters=args.iters + 1, capacity=128)
    T, E, k, H, I = w.tokens, w.n_experts, w.top_k, w.hidden, w.inter
    P = 16                                  # host blocks, aliased over the 128 experts
    t0 = time.time()
    pool = HN.fill_pool(w, args.seed, P)
    prof = oled.profile_mask("ffn_up", "ffn_down", "ffn_dense_up", "ffn_dense_down", "h2d",
                             "route_topk", "permute", "combine")
    ctx = HN.make_context(w, pool, capacity=E, n_layers=1, profile_ops=prof)
    lg = W.logits_block(w, args.seed, 0, 0)
    log(f"setup {time.time() - t0:.1f}s")
    y = torch.empty((T, H), dtype=torch.bfloat16, device="cuda")
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    layer_ms, ops, x_last = [], [], None
    for it in range(args.iters + 1):
        logits = torch.from_numpy(lg[it]).cuda()
        x = HN.to_device(W.activations(w, args.seed, 0, 0, it))
        conf = torch.from_numpy(W.confidence(w, args.seed, 0, it)).cuda()
        torch.cuda.synchronize()
        ctx.profile_collect()
        ev0.record()
        HN.layer_step(ctx, 0, logits, conf, x=x, y=y, report=False)
        ev1.record()
        torch.cuda.synchronize()
        if it > 0:                          # iteration 0 moves every expert in
            layer_ms.append(ev0.elapsed_time(ev1))
            ops += ctx.profile_collect()
        x_last = x
    st = ctx.read_layer_state(0, T)

    def agg(name):
        sel = [o for o in ops if o[0] == name]
        ms, fl, by = sum(o[2] for o in sel), sum(o[4] for o in sel), sum(o[3] for o in sel)
        return {"launches": len(sel), "avg_ms": round(ms / max(1, len(sel)), 4),
                "tflops": round(fl / 1e12 / (ms / 1e3), 1) if ms > 0 else None,
                "mfma_frac": round(fl / 1e12 / (ms / 1e3) / MFMA_BF16_PEAK_TFLOPS, 4)
                if ms > 0 else None,
                "flops_per_launch": int(fl / max(1, len(sel))),
                "bytes_per_launch": int(by / max(1, len(sel)))}

    up, down = agg("ffn_dense_up"), agg("ffn_dense_down")
    sel = [o for o in ops if o[0] in ("ffn_dense_up", "ffn_dense_down")]
    d_ms, d_fl = sum(o[2] for o in sel), sum(o[4] for o in sel)
    counts = st["counts"]

    # sampled rows of the last iteration against the oracle (float64)
    rows = np.random.default_rng(args.seed).choice(T, args.check_rows, replace=False)
    hbo = W.host_block_of(w, P)
    cache = {}

    def weights(e):
        b = int(hbo[e])
        if b not in cache:
            cache[b] = W.split_expert(w, O.decode(W.expert_block(w, args.seed, b)))
        return cache[b]

    idx, gates = O.route(lg[args.iters], k)
    xr = O.decode(W.activations(w, args.seed, 0, 0, args.iters))
    y_ref = O.moe_output(xr, idx, gates, weights, tokens=rows)
    y_got = O.decode(y.view(torch.int16).cpu().numpy().view(np.uint16))[rows]
    err = float(np.linalg.norm(y_got - y_ref) / np.linalg.norm(y_ref))
    ctx.close()
    pool.free()
    out = {
        "mode": "gemm",
        "config": {"workload": "prefill-like block: hidden 4096, 128 experts, top-8, expert "
                               "intermediate 1536, bf16, 16384 tokens (256 x 64), one layer, "
                               "all experts cached", "tokens": T, "routes": T * k},
        "rows_per_expert": {"min": int(counts.min()), "mean": float(counts.mean()),
                            "max": int(counts.max()), "dense_experts": int((counts >= 128).sum())},
        "dense_up": up, "dense_down": down,
        "dense_mfma_frac": round(d_fl / 1e12 / (d_ms / 1e3) / MFMA_BF16_PEAK_TFLOPS, 4)
        if d_ms > 0 else None,
        "streaming_launches": {"ffn_up": agg("ffn_up"), "ffn_down": agg("ffn_down")},
        "layer_ms": round(float(np.mean(layer_ms)), 3),
        "iterations": args.iters,
        "parity": {"rows": int(args.check_rows), "rel_l2": err, "tol": 2e-2, "ok": err <= 2e-2},
    }
    print(json.dumps(out), flush=True)
    if err > 2e-2:
        sys.exit(1)


def route(args):
    import torch
    from paper_2609_33385_amd import oled
    # 32 layers x 65535 tokens x 128 experts fp32 logits: 1 GiB over 32 launches
    # of each routing kernel (65535 is the largest block the priority sums allow)
    L, T, E, k, H, I = 32, 65535, 128, 8, 256, 256
    pool = oled.PinnedPool(E, 3 * H * I * 2)
    prof = oled.profile_mask("route_topk", "permute", "score_retain")
    ctx = oled.Context(H, I, E, k, L, E, T, "bf16", pool.ptr, pool.n_blocks,
                       np.tile(np.arange(E, dtype=np.int64), L), profile_ops=prof)
    g = torch.Generator(device="cuda")
    g.manual_seed(args.seed)
    logits = []
    for _ in range(L):   # per-sequence preference (64-token sequences) + token noise
        z = torch.randn((T + 63) // 64, E, generator=g, device="cuda").repeat_interleave(64, 0)[:T]
        logits.append(3.0 * z + torch.randn(T, E, generator=g, device="cuda"))
    conf = torch.rand(T, generator=g, device="cuda")
    torch.cuda.synchronize()
    s = torch.cuda.current_stream().cuda_stream
    ops = []
    t_wall = []
    for it in range(args.iters + 1):
        ctx.profile_collect()
        t0 = time.perf_counter()
        for l in range(L):
            ctx.route_block(l, logits[l].data_ptr(), T, s)
            ctx.apply_misses(l, report=False)
            ctx.score_and_retain(l, conf.data_ptr(), s)
        torch.cuda.synchronize()
        if it > 0:     # iteration 0 moves every expert in
            t_wall.append(time.perf_counter() - t0)
            ops += ctx.profile_collect()
    ctx.close()
    pool.free()

    # the same 1 GiB as one batch of 32 independent blocks: one top-k launch
    # over every token, the counting and ranking launches over (chunk, block),
    # and the priority numerators of every block (HIP events on the stream)
    lg_all = torch.stack(logits)
    del logits
    conf_all = torch.rand((L, T), generator=g, device="cuda")
    dev = dict(topk=torch.empty((L, T * k), dtype=torch.int32, device="cuda"),
               gates=torch.empty((L, T * k), dtype=torch.float32, device="cuda"),
               counts=torch.empty((L, E), dtype=torch.int32, device="cuda"),
               offsets=torch.empty((L, E + 1), dtype=torch.int32, device="cuda"),
               perm=torch.empty((L, T * k), dtype=torch.int32, device="cuda"),
               inv=torch.empty((L, T * k), dtype=torch.int32, device="cuda"),
               bad=torch.empty((L,), dtype=torch.int32, device="cuda"),
               S=torch.empty((L, E), dtype=torch.int64, device="cuda"))
    ws = torch.empty(oled.oled_route_batch_workspace(L, T, E), dtype=torch.uint8, device="cuda")
    st = torch.cuda.current_stream()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    t_route, t_prio = [], []
    for it in range(args.iters + 1):
        ev[0].record(st)
        rc = oled.oled_route_batch(lg_all, L, T, E, k, dev["topk"], dev["gates"], dev["counts"],
                                   dev["offsets"], dev["perm"], dev["inv"], dev["bad"], ws, st)
        ev[1].record(st)
        rc |= oled.oled_priority_batch(dev["topk"], dev["gates"], conf_all, L, T, E, k, dev["S"],
                                       None, st)
        ev[2].record(st)
        torch.cuda.synchronize()
        if rc:
            raise RuntimeError(oled.last_error(None))
        if it > 0:
            t_route.append(ev[0].elapsed_time(ev[1]))
            t_prio.append(ev[1].elapsed_time(ev[2]))
    assert int(dev["bad"].sum()) == 0

    def rate(ms, nbytes):
        gbs = nbytes / 1e9 / (ms / 1e3)
        return {"avg_us": round(ms * 1e3, 2), "bytes": nbytes, "GBps": round(gbs, 1),
                "hbm_frac": round(gbs / HBM_PEAK_GBS, 4)}

    # context: the read rate plain library reductions get on the same 1 GiB
    # (torch.amax over the experts of each token, the top-k's access pattern,
    # and a sum over the whole tensor)
    read_ref = {}
    for name, fn in (("amax_per_token", lambda: lg_all.amax(dim=2)),
                     ("sum_all", lambda: lg_all.sum())):
        for _ in range(2):
            fn()
        torch.cuda.synchronize()
        ts = []
        for _ in range(args.iters + 2):
            ev[0].record(st)
            fn()
            ev[1].record(st)
            torch.cuda.synchronize()
            ts.append(ev[0].elapsed_time(ev[1]))
        ms = float(np.mean(ts))
        gbs = L * T * E * 4 / 1e9 / (ms / 1e3)
        read_ref[name] = {"avg_us": round(ms * 1e3, 2), "GBps": round(gbs, 1),
                          "hbm_frac": round(gbs / HBM_PEAK_GBS, 4)}

    route_bytes = L * (T * E * 4 + T * k * 8 + T * k * 12 + E * 8)
    prio_bytes = L * (T * k * 8 + T * 4 + E * 8)
    batched = {"blocks": L, "calls": args.iters,
               "route_batch": rate(float(np.mean(t_route)), route_bytes),
               "priority_batch": rate(float(np.mean(t_prio)), prio_bytes)}

    def agg(name):
        sel = [o for o in ops if o[0] == name]
        ms, by = sum(o[2] for o in sel), sum(o[3] for o in sel)
        gbs = by / 1e9 / (ms / 1e3) if ms > 0 else 0.0
        return {"launches": len(sel), "avg_us": round(ms / max(1, len(sel)) * 1e3, 2),
                "bytes_per_launch": int(by / max(1, len(sel))), "GBps": round(gbs, 1),
                "hbm_frac": round(gbs / HBM_PEAK_GBS, 4)}

    out = {"mode": "route",
           "config": {"workload": "router logits of 32 layers x 65535 tokens x 128 experts fp32 "
                                  "(1 GiB per pass), top-8, all experts cached",
                      "layers": L, "tokens": T, "experts": E, "top_k": k,
                      "logit_bytes_per_pass": L * T * E * 4},
           "route_topk": agg("route_topk"), "permute": agg("permute"),
           "score_retain": agg("score_retain"), "passes": args.iters,
           "wall_ms_per_pass": round(float(np.mean(t_wall)) * 1e3, 3), "batched": batched,
           "torch_read_reference": read_ref}
    print(json.dumps(out), flush=True)


def gate(args):
    import torch
    from paper_2609_33385_amd import harness as HN
    from paper_2609_33385_amd import oled
    from paper_2609_33385_amd import workload as W
    out = {"mode": "gate", "shapes": []}
    for name, w in (("40% stack", W.WORKLOADS[2].replace(n_layers=1)),
                    ("batch 8", W.WORKLOADS[3].replace(n_layers=1)),
                    ("E=128 stack", W.WORKLOADS[4].replace(n_layers=1)),
                    ("prefill", W.WORKLOADS[5].replace(wid=400, batch=256, block=64, n_layers=1,
                                                      capacity=128))):
        T, E, H = w.tokens, w.n_experts, w.hidden
        pool = oled.PinnedPool(2, w.expert_bytes)
        ctx = HN.make_context(w, pool, capacity=0, profile_ops=oled.profile_mask("route_gemm"))
        x = HN.to_device(W.activations(w, args.seed, 0, 0, 0))
        g = HN.to_device(W.gate_weights(w, args.seed, 0))
        conf = torch.ones(T, device="cuda")
        s = torch.cuda.current_stream()
        ops = []
        for it in range(args.iters + 1):
            ctx.route_block_gate(0, x, g, T, s)
            ctx.apply_misses(0, report=False)
            ctx.score_and_retain(0, conf, s)
            torch.cuda.synchronize()
            got = ctx.profile_collect()
            if it > 0:
                ops += [o for o in got if o[0] == "route_gemm"]
        ctx.close()
        pool.free()
        ms = sum(o[2] for o in ops) / len(ops)
        by, fl = ops[0][3], ops[0][4]
        out["shapes"].append({"shape": name, "tokens": T, "hidden": H, "experts": E,
                              "avg_us": round(ms * 1e3, 2),
                              "TFLOPs": round(fl / 1e12 / (ms / 1e3), 2),
                              "GBps": round(by / 1e9 / (ms / 1e3), 1),
                              "hbm_frac": round(by / 1e9 / (ms / 1e3) / HBM_PEAK_GBS, 4),
                              "mfma_frac": round(fl / 1e12 / (ms / 1e3) / MFMA_BF16_PEAK_TFLOPS, 4),
                              "launches": len(ops)})
    print(json.dumps(out), flush=True)


def vendor(args):
    import torch
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    g = torch.Generator(device="cuda")
    g.manual_seed(args.seed)
    ops = {}
    out = {"mode": "vendor",
           "config": {"workload": "torch.bmm (hipBLASLt), bf16 in and out, contiguous operands: "
                                  "128 batches of 1024 x K by K x N"}}
    for name, (G, M, K, N) in (("gate_up", (128, 1024, 4096, 3072)),
                               ("down", (128, 1024, 1536, 4096))):
        a = torch.randn(G, M, K, generator=g, device="cuda").to(torch.bfloat16)
        b = torch.randn(G, K, N, generator=g, device="cuda").to(torch.bfloat16).contiguous()
        c = torch.empty(G, M, N, device="cuda", dtype=torch.bfloat16)
        for _ in range(3):
            torch.bmm(a, b, out=c)
        torch.cuda.synchronize()
        ms = []
        for _ in range(args.iters * 3):
            ev0.record()
            torch.bmm(a, b, out=c)
            ev1.record()
            torch.cuda.synchronize()
            ms.append(ev0.elapsed_time(ev1))
        fl = 2.0 * G * M * K * N
        avg = sum(ms) / len(ms)
        out[name] = {"dims": [G, M, K, N], "launches": len(ms), "avg_ms": round(avg, 4),
                     "tflops": round(fl / 1e12 / (avg / 1e3), 1),
                     "mfma_frac": round(fl / 1e12 / (avg / 1e3) / MFMA_BF16_PEAK_TFLOPS, 4)}
        ops[name] = (a, b, c, fl)
    # the down product right behind the gate/up product, as the layer runs them
    (ua, ub, uc, _), (da, db, dc, dfl) = ops["gate_up"], ops["down"]
    ev2 = torch.cuda.Event(enable_timing=True)
    ms = []
    for i in range(args.iters * 3 + 2):
        ev0.record()
        torch.bmm(ua, ub, out=uc)
        ev1.record()
        torch.bmm(da, db, out=dc)
        ev2.record()
        torch.cuda.synchronize()
        if i >= 2:
            ms.append(ev1.elapsed_time(ev2))
    avg = sum(ms) / len(ms)
    out["down_after_gate_up"] = {"launches": len(ms), "avg_ms": round(avg, 4),
                                 "mfma_frac": round(dfl / 1e12 / (avg / 1e3) /
                                                    MFMA_BF16_PEAK_TFLOPS, 4)}
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gemm", action="store_true")
    ap.add_argument("--route", action="store_true")
    ap.add_argument("--gate", action="store_true")
    ap.add_argument("--vendor", action="store_true")
    ap.add_argument("--iters", type=int, default=3)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--check-rows", type=int, default=8)
    args = ap.parse_args()
    import torch
    from paper_2609_33385_amd import oled
    torch.cuda.set_device(0)
    oled.load()
    if args.gemm:
        gemm(args)
    if args.route:
        route(args)
    if args.gate:
        gate(args)
    if args.vendor:
        vendor(args)


if __name__ == "__main__":
    main()
