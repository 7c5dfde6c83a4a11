"""GPU parity of route_block_gate (the gate GEMM in front of the routing):
the fp32 logits against the oracle's float64 logits within the fp32
accumulation bound; the whole control path, run on the GPU's own logits,
bit for bit against the oracle on the same logits; and, for every token
whose k-th and (k+1)-th exact logits are further apart than the rounding can
move them, the GPU's top-k set equals the exact one."""
import sys

import numpy as np
import pytest
import torch

from oracle import oled_oracle as O
from paper_2609_33385_amd import harness as HN
from paper_2609_33385_amd import oled
from paper_2609_33385_amd import workload as W

from gpu_common import compare_control

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    oled.load()


CASES = [
    ("bf16", 1, 32, 64, 8, 2048, 26),
    ("bf16", 25, 60, 128, 8, 4096, 51),
    ("f32", 1, 32, 8, 2, 256, 4),
    ("bf16", 17, 241, 200, 3, 512, 80),
    ("bf16", 3, 11, 16, 1, 128, 6),
]


@pytest.mark.parametrize("dtype,batch,block,E,k,H,C", CASES)
def test_gate_routing(dtype, batch, block, E, k, H, C):
    w = W.WORKLOADS[2].replace(wid=360, name=f"gate-{dtype}-E{E}-H{H}", dtype=dtype, batch=batch,
                               block=block, n_experts=E, top_k=k, hidden=H, inter=128, n_layers=2,
                               n_iters=2, capacity=C)
    T = w.tokens
    _say(f"[gate] {w.name} T={T} k={k}")
    pool = HN.fill_pool(w, 0, 4)
    ctx = HN.make_context(w, pool)
    s = torch.cuda.current_stream()
    res = [np.zeros(E, bool) for _ in range(2)]
    checked = 0
    try:
        for i in range(2):
            conf_h = W.confidence(w, 0, 0, i)
            conf = torch.from_numpy(conf_h).cuda()
            for l in range(2):
                xh = W.activations(w, 0, l, 0, i)
                gh = W.gate_weights(w, 0, l)
                x, g = HN.to_device(xh), HN.to_device(gh)
                ctx.route_block_gate(l, x, g, T, s)
                ctx.apply_misses(l, report=False)
                ctx.score_and_retain(l, conf, s)
                st = ctx.read_layer_state(l, T)
                lg = st["logits"]
                ref = O.router_logits(O.decode(xh), O.decode(gh))
                bound = O.fp32_sum_bound(O.decode(xh), O.decode(gh))
                err = np.abs(lg.astype(np.float64) - ref)
                assert np.all(err <= bound), f"logit error {err.max():.3e} above the bound"
                o = O.layer_step(lg.copy(), conf_h, res[l], k, C)
                o["lockstep"] = True
                o = compare_control(st, o, T, f"{w.name} l={l} i={i}", lg.copy(), conf_h, C)
                res[l] = o["resident_after"]
                # where rounding cannot reorder them, the exact top-k set
                srt = np.sort(ref, axis=1)[:, ::-1]
                if k < E:
                    tb = bound.max(axis=1)
                    safe = (srt[:, k - 1] - srt[:, k]) > 2 * tb
                    exact = np.argsort(-ref, axis=1, kind="stable")[:, :k]
                    for t in np.nonzero(safe)[0]:
                        assert set(exact[t]) == set(st["topk_idx"][t]), t
                    checked += int(safe.sum())
        _say(f"[gate] ok, exact top-k sets checked on {checked} token-layers")
    finally:
        ctx.close()
        pool.free()


# blocks large enough for the wide tiles of the gate GEMM (64 tokens x 128 or
# 64 experts per workgroup), with ragged token and expert tails, in both dtypes
TILE_CASES = [
    ("bf16", 40, 410, 128, 256),
    ("bf16", 3, 5481, 48, 256),
    ("f32", 40, 410, 128, 128),
    ("bf16", 40, 410, 64, 128),   # two of the four hidden-dimension parts are empty
]


@pytest.mark.parametrize("dtype,batch,block,E,H", TILE_CASES)
def test_gate_logits_wide_tiles(dtype, batch, block, E, H):
    w = W.WORKLOADS[2].replace(wid=361, name=f"gate-wide-{dtype}-E{E}-H{H}", dtype=dtype,
                               batch=batch, block=block, n_experts=E, top_k=4, hidden=H,
                               inter=128, n_layers=1, n_iters=1, capacity=E // 2)
    T = w.tokens
    _say(f"[gate wide] {w.name} T={T}")
    pool = HN.fill_pool(w, 0, 4)
    ctx = HN.make_context(w, pool)
    s = torch.cuda.current_stream()
    try:
        xh = W.activations(w, 1, 0, 0, 0)
        gh = W.gate_weights(w, 1, 0)
        x, g = HN.to_device(xh), HN.to_device(gh)
        conf = torch.from_numpy(W.confidence(w, 1, 0, 0)).cuda()
        ctx.route_block_gate(0, x, g, T, s)
        ctx.apply_misses(0, report=False)
        ctx.score_and_retain(0, conf, s)
        lg = ctx.read_layer_state(0, T)["logits"]
        ref = O.router_logits(O.decode(xh), O.decode(gh))
        bound = O.fp32_sum_bound(O.decode(xh), O.decode(gh))
        err = np.abs(lg.astype(np.float64) - ref)
        assert np.all(err <= bound), f"logit error {err.max():.3e} above the bound"
        _say(f"[gate wide] ok, max error {err.max():.3e}")
    finally:
        ctx.close()
        pool.free()


def test_gate_error_paths():
    """route_block_gate's argument and state checks, and a non-finite token
    row: its logits are non-finite, so the block is refused like a bad block
    of logits and the cache state does not change."""
    w = W.WORKLOADS[2].replace(wid=362, name="gate-errors", n_layers=2, n_iters=2, hidden=256,
                               inter=128, capacity=26)
    T, H = w.tokens, w.hidden
    pool = HN.fill_pool(w, 0, 4)
    ctx = HN.make_context(w, pool)
    s = torch.cuda.current_stream()
    try:
        xh = W.activations(w, 0, 0, 0, 0)
        x, g = HN.to_device(xh), HN.to_device(W.gate_weights(w, 0, 0))
        conf = torch.from_numpy(W.confidence(w, 0, 0, 0)).cuda()
        assert oled.route_block_gate(ctx.ctx, 0, None, g, T, s) == oled.OLED_ERR_INVALID_ARG
        assert oled.route_block_gate(ctx.ctx, 0, x, None, T, s) == oled.OLED_ERR_INVALID_ARG
        assert oled.route_block_gate(ctx.ctx, 0, x, g, 0, s) == oled.OLED_ERR_INVALID_ARG
        assert oled.route_block_gate(ctx.ctx, 0, x, g, T + 1, s) == oled.OLED_ERR_INVALID_ARG
        assert oled.route_block_gate(ctx.ctx, 2, x, g, T, s) == oled.OLED_ERR_INVALID_ARG
        # a good layer fills the cache
        ctx.route_block_gate(0, x, g, T, s)
        # in flight: a second routing of any layer is out of order
        assert oled.route_block_gate(ctx.ctx, 1, x, g, T, s) == oled.OLED_ERR_STATE
        ctx.apply_misses(0, report=False)
        ctx.score_and_retain(0, conf, s)
        before = ctx.read_layer_state(0, T)["resident_after"].copy()
        assert before.any()
        # a NaN in one token row
        bad = x.clone()
        bad[5, 7] = float("nan")
        ctx.route_block_gate(0, bad, g, T, s)
        rep = oled.MissReport()
        assert oled.apply_misses(ctx.ctx, 0, None, rep) == oled.OLED_ERR_INVALID_ARG
        assert np.array_equal(ctx.read_layer_state(0, T)["resident_after"], before)
        _say("[gate errors] ok")
    finally:
        ctx.close()
        pool.free()
