"""GPU parity at large blocks, where routing takes one token per lane, the
permutation runs over many workgroups (counting launch + ranking launch) and
the priority numerators are summed by several workgroups: the largest block
(65535 tokens), ragged chunk tails, top-k below the kernel's list length,
expert counts that are not a multiple of the 32-expert LDS chunk, and fp32.
Control path bit for bit against the oracle at every layer-iteration; layer
outputs on sampled token rows."""
import sys

import numpy as np
import pytest
import torch

from oracle import oled_oracle as O
from paper_2609_33385_amd import harness as HN
from paper_2609_33385_amd import oled
from paper_2609_33385_amd import workload as W

from gpu_common import (LockstepOracle, OracleWeights, compare_control, rel_l2, run_schedule_gpu,
                        tol)

pytestmark = pytest.mark.gpu

BASE = W.WORKLOADS[2].replace(n_experts=128, top_k=8, hidden=256, inter=256, n_layers=2, n_iters=3,
                              capacity=51)


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    oled.load()


def _run(w, seed, forward=False, out_rows=16):
    layers = list(range(w.n_layers))
    _say(f"[large] {w.name} T={w.tokens} E={w.n_experts} k={w.top_k} {w.dtype} C={w.capacity} "
         f"forward={forward}")
    # one host block per (layer, expert) where the weights are small enough,
    # else E + 1 (distinct within a layer, shifted per layer)
    P = len(layers) * w.n_experts if w.expert_bytes * len(layers) * w.n_experts <= (1 << 30) \
        else w.n_experts + 1
    lock = LockstepOracle(len(layers), w.n_experts, w.top_k, w.capacity)
    raw = W.expert_blocks(w, seed, range(P))
    pool = HN.fill_pool(w, seed, P, raw=raw)
    ctx = HN.make_context(w, pool)
    ow = OracleWeights(w, seed, P, len(layers), raw=raw)
    rows = np.random.default_rng(seed).choice(w.tokens, min(out_rows, w.tokens), replace=False)
    worst = [0.0]

    def check(i, li, st, y, rep):
        o = lock.step(li, W.logits(w, seed, layers[li], 0, i), W.confidence(w, seed, 0, i), st,
                      f"{w.name} l={li} i={i}")
        if y is not None:
            x = O.decode(W.activations(w, seed, layers[li], 0, i))
            y_ref = O.moe_output(x, o["idx"], o["gates"], ow.fn(li), tokens=rows)
            err = rel_l2(O.decode(y)[rows], y_ref)
            worst[0] = max(worst[0], err)
            assert err <= tol(w), f"l={li} i={i}: rel L2 {err:.3e}"

    try:
        run_schedule_gpu(ctx, w, seed, layers, w.n_iters, forward, check)
    finally:
        ctx.close()
        pool.free()
    _say(f"[large] ok, worst rel L2 {worst[0]:.3e}")


def test_largest_block_control_path():
    _run(BASE.replace(wid=320, name="t65535", batch=255, block=257), 0)


@pytest.mark.parametrize("E,k,batch,block", [(128, 8, 17, 241), (64, 6, 9, 130), (200, 3, 5, 411),
                                              (40, 1, 3, 700)])
def test_ragged_blocks_forward(E, k, batch, block):
    w = BASE.replace(wid=321, name=f"e{E}k{k}t{batch * block}", n_experts=E, top_k=k, batch=batch,
                     block=block, capacity=int(0.4 * E))
    _run(w, 1, forward=True)


def test_large_block_f32():
    w = BASE.replace(wid=322, name="f32-t3000", dtype="f32", batch=12, block=250, capacity=40)
    _run(w, 2, forward=True)


@pytest.mark.parametrize("E,k", [(128, 8), (64, 4), (200, 2), (33, 16)])
def test_lane_routing_ties(E, k):
    """Large-block routing on logits full of exact ties (values on a 0.5 grid,
    signed zeros) and near ties (one ulp apart, so their packed keys agree in
    their top 24 bits): those tokens take the exact re-ranking; every route and
    gate bit for bit against the oracle."""
    T = 2100
    w = BASE.replace(wid=323, name=f"lane-ties-e{E}k{k}", n_experts=E, top_k=k, batch=7, block=300,
                     n_layers=1, n_iters=1, capacity=E // 3)
    assert w.tokens == T
    rng = np.random.default_rng(50 + E + k)
    lg = (np.round(rng.standard_normal((T, E)) * 2) / 2).astype(np.float32)
    nudge = rng.uniform(0, 1, (T, E)) < 0.25
    lg = np.where(nudge, np.nextafter(lg, np.float32(np.inf)), lg).astype(np.float32)
    zero = (lg == 0) & (rng.uniform(0, 1, (T, E)) < 0.5)
    lg[zero] = np.float32(-0.0)
    _say(f"[lane ties] E={E} k={k} T={T}")
    pool = HN.fill_pool(w, 0, 4)
    ctx = HN.make_context(w, pool)
    s = torch.cuda.current_stream()
    try:
        conf = torch.from_numpy(W.confidence(w, 0, 0, 0)).cuda()
        ctx.route_block(0, torch.from_numpy(lg).cuda(), T, s)
        ctx.apply_misses(0, report=False)
        ctx.score_and_retain(0, conf, s)
        st = ctx.read_layer_state(0, T)
        idx_ref, g_ref = O.route(lg, k)
        bad = np.nonzero(np.any(st["topk_idx"] != idx_ref, axis=1))[0]
        assert bad.size == 0, f"tokens {bad[:5]} routed differently"
        o = O.layer_step(lg, W.confidence(w, 0, 0, 0), np.zeros(E, bool), k, w.capacity)
        compare_control(st, o, T, f"lane ties E={E} k={k}", lg, W.confidence(w, 0, 0, 0),
                        w.capacity)
        _say("[lane ties] ok")
    finally:
        ctx.close()
        pool.free()
