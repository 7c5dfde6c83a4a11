"""Retention-policy comparison on one MI355X (the paper's mechanism analysis,
Sec. 5.3, on synthetic traces).

For the 40%-residency layer stack (bf16, hidden 2048, 64 experts, top-8,
intermediate 1024, 16 layers, 32 tokens per iteration, 8 iterations per
block) and variants of it, runs blocks of denoising iterations through the
whole hot path (routing, cached and transferred experts, combine, retention)
under each retention policy: the paper's confidence-gate priority, LRU and
LFU, and the priority with layer-adaptive sizing. Reports per run the expert
cache utilisation (hits / C per layer-iteration), the clairvoyant ideal
bound min(C, |A|) / C, misses per layer-iteration, the effective transfer
ratio (transferred experts retained and activated again at the layer's next
iteration) and layer-tokens/s. The first block (cold cache) is excluded.

Variants: "plain" (iteration noise independent of confidence), "informed"
(a token's routing noise scaled by 2 (1 - its confidence), so confident
tokens keep their experts, as the paper observes), "hetero" (layers with
different routing spread), each at 13 (20%) and 26 (40%) experts per layer.

Prints one JSON line per run; inputs are seeded and synthetic.
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


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--blocks", type=int, default=4)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--variants", default="plain,informed,hetero")
    ap.add_argument("--capacities", default="13,26")
    args = ap.parse_args()

    import torch
    from bench import fill_pool_device, make_inputs
    from paper_2609_33385_amd import oled
    from paper_2609_33385_amd import workload as W

    torch.cuda.set_device(0)
    lib = oled.load()
    base = W.WORKLOADS[2]
    variants = {"plain": base, "informed": base.replace(conf_informed=True),
                "hetero": base.replace(sigma_s_layers=(0.5, 1.0, 1.5, 2.0, 2.5, 3.0, 4.0, 5.0))}
    L, T, E = base.n_layers, base.tokens, base.n_experts
    pool = oled.PinnedPool(L * E, base.expert_bytes)
    fill_pool_device(pool, base, args.seed)
    n_steps = args.blocks * base.n_iters
    s = torch.cuda.current_stream()
    sp = s.cuda_stream
    y = torch.empty((T, base.hidden), dtype=torch.bfloat16, device="cuda")
    for vname in args.variants.split(","):
        w = variants[vname]
        t0 = time.time()
        logits, xs, conf = make_inputs(w, args.seed, n_steps)
        log(f"{vname}: inputs {time.time() - t0:.1f}s")
        for C in (int(c) for c in args.capacities.split(",")):
            runs = [("priority", 0), ("lru", 0), ("lfu", 0), ("priority", 5)]
            for policy, period in runs:
                ctx = oled.Context(w.hidden, w.inter, E, w.top_k, L, C, T, w.dtype, pool.ptr,
                                   pool.n_blocks, W.host_block_of(w, pool.n_blocks),
                                   policy=policy, adapt_period=period)
                h = ctx.ctx
                acc = dict(hits=0, misses=0, active=0, ideal=0, li=0, moved=0, reused=0, cap=0)
                elapsed = 0.0
                for g in range(n_steps):
                    torch.cuda.synchronize()
                    t1 = time.perf_counter()
                    for l in range(L):
                        lib.route_block(h, l, logits[g, l].data_ptr(), T, sp)
                        lib.moe_forward_cached(h, l, xs[g, l].data_ptr(), y.data_ptr(), sp)
                        lib.apply_misses(h, l, None, None)
                        lib.score_and_retain(h, l, conf[g].data_ptr(), sp)
                    torch.cuda.synchronize()
                    dt = time.perf_counter() - t1
                    caps = [ctx.read_layer_state(l)["capacity"] for l in range(L)] if period else None
                    st = ctx.collect_stats()
                    if g < base.n_iters:      # first block: cold cache
                        continue
                    elapsed += dt
                    acc["hits"] += st["n_hits"]
                    acc["misses"] += st["n_misses"]
                    acc["active"] += st["n_active"]
                    acc["li"] += st["layer_iters"]
                    acc["moved"] += st["n_prev_transferred"]
                    acc["reused"] += st["n_transfers_reused"]
                    acc["ideal"] += st["n_ideal_hits"]
                err = oled.last_error(h)
                ctx.close()
                li = max(1, acc["li"])
                out = {"variant": vname, "capacity": C, "policy": policy, "adapt_period": period,
                       "util": round(acc["hits"] / (C * li), 4),
                       "ideal_util": round(acc["ideal"] / (C * li), 4),
                       "misses_per_layer_iter": round(acc["misses"] / li, 3),
                       "active_per_layer_iter": round(acc["active"] / li, 3),
                       "effective_transfer_ratio": round(acc["reused"] / max(1, acc["moved"]), 4),
                       "layer_tokens_per_s": round(acc["li"] * T / elapsed, 1) if elapsed else None,
                       "timed_layer_iters": acc["li"]}
                if caps is not None:
                    out["capacities_end"] = caps
                if err:
                    out["error"] = err
                print(json.dumps(out), flush=True)
    pool.free()


if __name__ == "__main__":
    main()
