"""GPU parity of the HIP path (through the C ABI) against the CPU oracle.

Integer results (routing indices, permutation, counts, hits/misses, priority
numerators, retained sets) and the fp32 gates must match bit for bit; layer
outputs within relative L2 1e-5 (fp32) or 2e-2 (bf16). Every read of a
layer's state also checks slot conservation over the device cache state.
Both transfers of the misses are covered: workgroups of the hit launches
("shader", the default) and hipMemcpyAsync on a copy stream ("sdma").
"""
import sys

import numpy as np
import pytest
import torch

from oracle import oled_oracle as O
from paper_2609_33385_amd import harness as HN
from paper_2609_33385_amd import oled
from paper_2609_33385_amd import workload as W

from gpu_common import (LockstepOracle, OracleWeights, check_report, compare_control,
                        oracle_schedule, rel_l2, run_schedule_gpu, tol)

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    oled.load()


def _chain(w, seed, layers, n_iters, n_blocks, out_at=None, out_tokens=None, capacity=None,
           forward=True, copy_mode="shader", report=True, expect_dense=False):
    """Runs a schedule on both sides and compares every layer-iteration, the
    oracle advancing in lockstep with the GPU.

    n_blocks: host pool blocks; expert (l, e) of the chain reads block
    (l*E + e) mod n_blocks, so n_blocks >= len(layers)*E gives every tested
    expert weights of its own, and E + 1 gives distinct weights within a
    layer that shift from layer to layer.
    out_at: set of (layer index, iteration) whose outputs are checked (None: all).
    out_tokens: token rows checked there (None: all).
    """
    C = w.capacity if capacity is None else capacity
    _say(f"[chain] {w.name} layers={list(layers)} iters={n_iters} C={C} P={n_blocks} "
         f"copy={copy_mode} report={report}")
    raw = W.expert_blocks(w, seed, range(n_blocks))
    pool = HN.fill_pool(w, seed, n_blocks, raw=raw)
    prof = oled.profile_mask("ffn_dense_up", "ffn_dense_down") if expect_dense else 0
    ctx = HN.make_context(w, pool, capacity=C, n_layers=len(layers), copy_mode=copy_mode,
                          profile_ops=prof)
    lock = LockstepOracle(len(layers), w.n_experts, w.top_k, C)
    ow = OracleWeights(w, seed, n_blocks, len(layers), raw=raw)
    worst = [0.0]

    def check(i, li, st, y, rep):
        where = f"{w.name} l={layers[li]} i={i}"
        o = lock.step(li, W.logits(w, seed, layers[li], 0, i), W.confidence(w, seed, 0, i),
                      st, where)
        check_report(rep, o, w.expert_bytes, where)
        if y is None or (out_at is not None and (li, i) not in out_at):
            return
        x = O.decode(W.activations(w, seed, layers[li], 0, i))
        rows = np.arange(w.tokens) if out_tokens is None else np.asarray(out_tokens)
        y_ref = O.moe_output(x, o["idx"], o["gates"], ow.fn(li), tokens=rows)
        err = rel_l2(O.decode(y)[rows], y_ref)
        worst[0] = max(worst[0], err)
        assert err <= tol(w), f"{where}: rel L2 {err:.3e} > {tol(w)}"

    try:
        run_schedule_gpu(ctx, w, seed, layers, n_iters, forward, check, report=report)
        if expect_dense:   # the dense-tile launches ran, with work
            ops = ctx.profile_collect()
            for name in ("ffn_dense_up", "ffn_dense_down"):
                assert any(o[0] == name and o[4] > 0 for o in ops), f"{w.name}: no {name} launch"
    finally:
        ctx.close()
        pool.free()
    _say(f"[chain] {w.name} ok, worst rel L2 {worst[0]:.3e}, accepted gate roundings "
         f"{lock.flips}")


@pytest.mark.parametrize("copy_mode", ["shader", "sdma"])
def test_cfg1_full_schedule(copy_mode):
    w = W.WORKLOADS[1]
    _chain(w, 0, range(w.n_layers), w.n_iters, w.n_layers * w.n_experts, copy_mode=copy_mode)


def test_cfg1_control_path_without_reports():
    """No forward and no reports: only the transfer-only launch moves misses."""
    w = W.WORKLOADS[1]
    _chain(w, 0, range(w.n_layers), w.n_iters, 8, forward=False, report=False)


SMALL = [  # (E, k, T, C, dtype, H, I)
    (1, 1, 1, 0, "f32", 128, 128),
    (5, 2, 37, 2, "f32", 128, 256),
    (64, 8, 65, 26, "bf16", 256, 128),
    (128, 8, 200, 51, "bf16", 128, 384),
    (256, 16, 33, 100, "bf16", 128, 128),
    (33, 3, 600, 33, "f32", 128, 128),
    (64, 8, 130, 0, "bf16", 256, 256),
    (16, 4, 1025, 40, "bf16", 128, 128),
    (128, 16, 64, 51, "bf16", 128, 128),   # largest block routed by the fused path
    (128, 8, 64, 51, "f32", 256, 1024),    # down GEMM with its K split in two
]


@pytest.mark.parametrize("E,k,T,C,dt,H,I", SMALL)
def test_small_shapes(E, k, T, C, dt, H, I):
    w = W.WORKLOADS[1].replace(wid=100 + E, name=f"small-E{E}-k{k}-T{T}", dtype=dt, batch=1,
                               block=T, n_experts=E, top_k=k, hidden=H, inter=I, n_layers=2,
                               n_iters=3, capacity=C)
    _chain(w, 1, range(2), 3, 2 * E)
    if E in (5, 64):
        _chain(w, 1, range(2), 3, 2 * E, copy_mode="sdma")


def test_ties_and_signed_zero():
    """Tied logits (small integer alphabet) and -0.0 / +0.0 through the ABI."""
    rng = np.random.default_rng(5)
    E, k, T, H, I = 12, 3, 70, 128, 128
    w = W.WORKLOADS[1].replace(wid=200, name="ties", batch=1, block=T, n_experts=E, top_k=k,
                               hidden=H, inter=I, n_layers=1, n_iters=1, capacity=4)
    lg = rng.integers(-2, 3, size=(T, E)).astype(np.float32)
    lg[::5, 0] = -0.0
    lg[::5, 1] = 0.0
    conf = rng.uniform(0, 1, T).astype(np.float32)
    pool = HN.fill_pool(w, 0, E)
    ctx = HN.make_context(w, pool)
    try:
        HN.layer_step(ctx, 0, torch.from_numpy(lg).cuda(), torch.from_numpy(conf).cuda())
        st = ctx.read_layer_state(0, T)
        ref = O.layer_step(lg, conf, np.zeros(E, bool), k, 4)
        compare_control(st, ref, T, "ties", lg, conf, 4)
    finally:
        ctx.close()
        pool.free()


@pytest.mark.parametrize("copy_mode", ["shader", "sdma"])
def test_cfg2_chain(copy_mode):
    """All 16 layers; E + 1 host blocks: distinct weights within every layer,
    shifted from layer to layer."""
    w = W.WORKLOADS[2]
    L, N = w.n_layers, w.n_iters
    out_at = {(l, i) for l in (0, L // 2, L - 1) for i in (0, 1, N - 1)}
    _chain(w, 0, range(L), N, w.n_experts + 1, out_at=out_at, copy_mode=copy_mode)


def test_cfg2_chain_unaliased():
    """Four layers, one host block per (layer, expert): no two tested experts
    share weights, so a slot, address or work-item mistake that reads another
    expert's weights changes the output."""
    w = W.WORKLOADS[2]
    layers, N = [0, 5, 10, 15], w.n_iters
    out_at = {(li, i) for li in range(4) for i in (1, N - 1)}
    _chain(w, 0, layers, N, len(layers) * w.n_experts, out_at=out_at)


def test_cfg2_no_sync_until_the_end():
    """The bench's call pattern: no report and no host read between layers.
    Every output, the final resident sets and the routing totals against the
    oracle."""
    w = W.WORKLOADS[2]
    layers, N, T = [0, 5, 11, 15], w.n_iters, w.tokens
    _say(f"[async] {w.name} layers={layers} iters={N}")
    P = len(layers) * w.n_experts
    raw = W.expert_blocks(w, 0, range(P))
    pool = HN.fill_pool(w, 0, P, raw=raw)
    ctx = HN.make_context(w, pool, n_layers=len(layers))
    ref = oracle_schedule(w, 0, layers, N, w.capacity)
    ow = OracleWeights(w, 0, P, len(layers), raw=raw)
    s = torch.cuda.current_stream()
    dt = HN.torch_dtype(w)
    try:
        ins = []
        for i in range(N):
            conf = torch.from_numpy(W.confidence(w, 0, 0, i)).cuda()
            for li, l in enumerate(layers):
                lg = torch.from_numpy(W.logits(w, 0, l, 0, i)).cuda()
                x = HN.to_device(W.activations(w, 0, l, 0, i))
                ins.append((i, li, lg, conf, x, torch.empty((T, w.hidden), dtype=dt, device="cuda")))
        torch.cuda.synchronize()
        for i, li, lg, conf, x, y in ins:
            HN.layer_step(ctx, li, lg, conf, x, y, stream=s, report=False)
        stats = ctx.collect_stats()
        for li in range(len(layers)):
            st = ctx.read_layer_state(li, T)
            np.testing.assert_array_equal(st["resident_after"], ref[N - 1][li]["resident_after"])
        flat = [ref[i][li] for i in range(N) for li in range(len(layers))]
        assert stats["layer_iters"] == N * len(layers)
        assert stats["n_hits"] == sum(o["n_hits"] for o in flat)
        assert stats["n_misses"] == sum(o["n_misses"] for o in flat)
        assert stats["n_active"] == sum(o["n_active"] for o in flat)
        assert stats["h2d_bytes"] == stats["n_misses"] * w.expert_bytes
        worst = 0.0
        for i, li, lg, conf, x, y in ins:
            if (i, li) not in {(0, 0), (1, 2), (N - 1, 3), (N // 2, 1)}:
                continue
            o = ref[i][li]
            xx = O.decode(W.activations(w, 0, layers[li], 0, i))
            y_ref = O.moe_output(xx, o["idx"], o["gates"], ow.fn(li))
            err = rel_l2(O.decode(HN.from_device(y)), y_ref)
            worst = max(worst, err)
            assert err <= tol(w), f"l={layers[li]} i={i}: rel L2 {err:.3e}"
        _say(f"[async] ok, worst rel L2 {worst:.3e}")
    finally:
        ctx.close()
        pool.free()


def test_cfg3_chain():
    w = W.WORKLOADS[3]
    L, N = w.n_layers, w.n_iters
    _chain(w, 0, range(L), N, w.n_experts + 1, out_at={(0, 0), (L - 1, N - 1)})


@pytest.mark.parametrize("wid", [4, 5])
def test_cfg45_chain(wid):
    """The E=128 stacks on three sampled layers, one host block per (layer,
    expert) (384 blocks of 36 MiB): no two tested experts share weights."""
    w = W.WORKLOADS[wid]
    layers = [0, w.n_layers // 2, w.n_layers - 1]
    rows = np.random.default_rng(wid).choice(w.tokens, 16, replace=False)
    _chain(w, 0, layers, w.n_iters, len(layers) * w.n_experts,
           out_at={(0, 0), (1, 1), (2, w.n_iters - 1)}, out_tokens=rows)


DENSE = W.WORKLOADS[1].replace(wid=300, name="dense", dtype="bf16", batch=4, block=256,
                               n_experts=16, top_k=4, hidden=512, inter=256, n_layers=2,
                               n_iters=3, capacity=6)


@pytest.mark.parametrize("copy_mode", ["shader", "sdma"])
def test_dense_tiles(copy_mode):
    """Experts with 128+ routed rows run as dense tiles: this block has experts
    with two 256-row items, one plus a shorter item, exactly 256 rows, a short
    item only, and fewer than 128 rows (streaming), as hits and as misses."""
    _chain(DENSE, 1, range(2), 3, 32, copy_mode=copy_mode, expect_dense=True)


@pytest.mark.parametrize("H,I", [(256, 512), (768, 1280)])
def test_dense_tiles_stage_counts(H, I):
    """Dense tiles whose K loops have 4 stages (gate/up at hidden 256: only the
    last four stages), 8, 12 (gate/up at hidden 768: one pass of the steady
    loop) and 20 (down at intermediate 1280), each against the oracle on
    sampled token rows, as hits and as misses."""
    w = DENSE.replace(wid=310 + H // 256, name=f"dense-H{H}-I{I}", hidden=H, inter=I)
    rows = np.random.default_rng(H + I).choice(w.tokens, 96, replace=False)
    _chain(w, 2, range(2), 3, 2 * w.n_experts + 1, out_at={(0, 0), (1, 1), (0, 2)},
           out_tokens=rows, expect_dense=True)


def test_dense_tiles_cross_residency_bitwise():
    """The dense / streaming split depends on the routed rows only, so outputs
    stay identical across cache states and transfers."""
    w = DENSE
    pool = HN.fill_pool(w, 1, 32)
    outs = {}
    for C, mode in ((w.n_experts, "shader"), (w.capacity, "shader"), (0, "shader"),
                    (w.capacity, "sdma")):
        ctx = HN.make_context(w, pool, capacity=C, n_layers=2, copy_mode=mode)
        got = []
        run_schedule_gpu(ctx, w, 1, range(2), 3, True,
                         lambda i, li, st, y, rep: got.append(y.copy()))
        ctx.close()
        outs[(C, mode)] = got
    pool.free()
    base = outs[(w.n_experts, "shader")]
    for key, got in outs.items():
        for y0, y1 in zip(base, got):
            assert np.array_equal(y0, y1), f"{key}: outputs differ from full residency"


def test_cross_residency_bitwise():
    """Outputs do not depend on the cache state or the transfer (lossless):
    C = E, 40% and 0 with the shader transfer, 40% with the copy engine."""
    w = W.WORKLOADS[2]
    layers, N = [0, 1], 4
    pool = HN.fill_pool(w, 0, 16)
    outs = {}
    for C, mode in ((w.n_experts, "shader"), (w.capacity, "shader"), (0, "shader"),
                    (w.capacity, "sdma")):
        ctx = HN.make_context(w, pool, capacity=C, n_layers=len(layers), copy_mode=mode)
        got = []
        run_schedule_gpu(ctx, w, 0, layers, N, True,
                         lambda i, li, st, y, rep: got.append((st["n_hits"], y.copy())))
        ctx.close()
        outs[(C, mode)] = got
    pool.free()
    base = outs[(w.n_experts, "shader")]
    for key, got in outs.items():
        for (h0, y0), (h1, y1) in zip(base, got):
            assert np.array_equal(y0, y1), f"{key}: outputs differ from full residency"
    assert sum(h for h, _ in outs[(0, "shader")]) == 0


@pytest.mark.parametrize("copy_mode", ["shader", "sdma"])
def test_error_paths(copy_mode):
    w = W.WORKLOADS[1]
    pool = HN.fill_pool(w, 0, 8)
    ctx = HN.make_context(w, pool, copy_mode=copy_mode)
    T, E = w.tokens, w.n_experts
    s = torch.cuda.current_stream()
    try:
        lg = torch.from_numpy(W.logits(w, 0, 0, 0, 0)).cuda()
        conf = torch.from_numpy(W.confidence(w, 0, 0, 0)).cuda()
        # out of order
        assert oled.apply_misses(ctx.ctx, 0, None, None) == oled.OLED_ERR_STATE
        assert oled.score_and_retain(ctx.ctx, 0, conf, s) == oled.OLED_ERR_STATE
        assert oled.route_block(ctx.ctx, 0, lg, 0, s) == oled.OLED_ERR_INVALID_ARG
        assert oled.route_block(ctx.ctx, 0, lg, T + 1, s) == oled.OLED_ERR_INVALID_ARG
        assert oled.route_block(ctx.ctx, 5, lg, T, s) == oled.OLED_ERR_INVALID_ARG
        # one good step fills the cache
        HN.layer_step(ctx, 0, lg, conf)
        before = ctx.read_layer_state(0, T)["resident_after"].copy()
        assert before.any()
        # a non-finite logit: apply_misses refuses, nothing changes
        bad = lg.clone()
        bad[3, 2] = float("nan")
        ctx.route_block(0, bad, T, s)
        rep = oled.MissReport()
        assert oled.apply_misses(ctx.ctx, 0, None, rep) == oled.OLED_ERR_INVALID_ARG
        assert np.array_equal(ctx.read_layer_state(0, T)["resident_after"], before)
        # confidence outside [0, 1]: retention rejected, R kept, reported
        lg1 = torch.from_numpy(W.logits(w, 0, 0, 0, 1)).cuda()
        badc = conf.clone()
        badc[0] = 1.5
        HN.layer_step(ctx, 0, lg1, badc)
        st = ctx.read_layer_state(0, T)
        assert st["rejected"]
        assert np.array_equal(st["resident_after"], before)
        ctx.route_block(0, lg1, T, s)
        rep = ctx.apply_misses(0)
        assert rep.rejected_layer == 0   # reported once, by the next apply_misses
        ctx.score_and_retain(0, conf, s)
        assert not ctx.read_layer_state(0, T)["rejected"]
    finally:
        ctx.close()
        pool.free()


def test_bad_block_without_report():
    """A non-finite logit with nobody asking for a report: nothing is staged,
    the retention commits nothing, and the next read of the layer says so once."""
    w = W.WORKLOADS[1]
    pool = HN.fill_pool(w, 0, 8)
    ctx = HN.make_context(w, pool)
    T = w.tokens
    s = torch.cuda.current_stream()
    try:
        lg = torch.from_numpy(W.logits(w, 0, 0, 0, 0)).cuda()
        conf = torch.from_numpy(W.confidence(w, 0, 0, 0)).cuda()
        HN.layer_step(ctx, 0, lg, conf, report=False)
        before = ctx.read_layer_state(0, T)["resident_after"].copy()
        bad = torch.from_numpy(W.logits(w, 0, 0, 0, 1)).cuda()
        bad[7, 1] = float("inf")
        x = HN.to_device(W.activations(w, 0, 0, 0, 1))
        y = torch.empty((T, w.hidden), dtype=torch.float32, device="cuda")
        HN.layer_step(ctx, 0, bad, conf, x, y, report=False)
        st = ctx.read_layer_state(0, T)
        assert st["rejected"]                                  # reported once
        assert np.array_equal(st["resident_after"], before)
        assert not ctx.read_layer_state(0, T)["rejected"]
        assert ctx.collect_stats()["n_bad_blocks"] == 1
    finally:
        ctx.close()
        pool.free()


def test_block_boundaries():
    """Blocks follow each other without resetting the caches (semi-autoregressive
    decoding, Sec. 2.1): two blocks of the 40% stack back to back, the second
    starting from the first block's resident sets; every layer-iteration
    against the oracle, outputs at the block boundary."""
    w = W.WORKLOADS[2]
    layers, N = [0, 7, 15], w.n_iters
    _say(f"[blocks] {w.name} layers={layers} blocks=2 iters={N}")
    P = len(layers) * w.n_experts
    raw = W.expert_blocks(w, 0, range(P))
    pool = HN.fill_pool(w, 0, P, raw=raw)
    ctx = HN.make_context(w, pool, n_layers=len(layers))
    lock = LockstepOracle(len(layers), w.n_experts, w.top_k, w.capacity)
    ow = OracleWeights(w, 0, P, len(layers), raw=raw)
    dt = HN.torch_dtype(w)
    try:
        for g in range(2 * N):
            b, i = divmod(g, N)
            conf = torch.from_numpy(W.confidence(w, 0, b, i)).cuda()
            for li, l in enumerate(layers):
                lg_h = W.logits(w, 0, l, b, i)
                lg = torch.from_numpy(lg_h).cuda()
                x = HN.to_device(W.activations(w, 0, l, b, i))
                y = torch.empty((w.tokens, w.hidden), dtype=dt, device="cuda")
                rep = HN.layer_step(ctx, li, lg, conf, x, y)
                st = ctx.read_layer_state(li, w.tokens)
                where = f"block {b} iter {i} layer {l}"
                o = lock.step(li, lg_h, W.confidence(w, 0, b, i), st, where)
                check_report(rep, o, w.expert_bytes, where)
                if g in (N - 1, N):
                    y_ref = O.moe_output(O.decode(W.activations(w, 0, l, b, i)), o["idx"],
                                         o["gates"], ow.fn(li))
                    err = rel_l2(O.decode(HN.from_device(y)), y_ref)
                    assert err <= tol(w), f"{where}: rel L2 {err:.3e}"
        _say("[blocks] ok")
    finally:
        ctx.close()
        pool.free()
