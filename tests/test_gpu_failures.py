"""Host-side failure handling of the runtime on the GPU, forced from the host
(oled_set_fault_injection): no kernel faults or hangs; every launch runs
normally.

* A miss copy that cannot be enqueued (copy-engine transfer): apply_misses
  returns OLED_ERR_HIP, the staged misses give their slots back, the layer's
  resident set and slot table are unchanged (slot conservation is checked at
  the state read), and the context goes on: the next iterations match the
  oracle replayed without the failed layer-iteration.
* A wait past its deadline: apply_misses returns OLED_ERR_HIP, the context
  refuses further layers until oled_reset_cache, after which a cold run
  matches the oracle again.
"""
import sys

import numpy as np
import pytest
import torch

from oracle import oled_oracle as O
from paper_2609_33385_amd import harness as HN
from paper_2609_33385_amd import oled
from paper_2609_33385_amd import workload as W

from gpu_common import LockstepOracle, OracleWeights, compare_control, rel_l2, tol

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    oled.load()


W2 = W.WORKLOADS[2].replace(n_layers=2, n_iters=4, capacity=8)


def _inputs(w, layer, it):
    lg = W.logits(w, 0, layer, 0, it)
    conf = W.confidence(w, 0, 0, it)
    x = W.activations(w, 0, layer, 0, it)
    return lg, conf, x


def _step(ctx, w, layer, it, y):
    lg, conf, x = _inputs(w, layer, it)
    return HN.layer_step(ctx, layer, torch.from_numpy(lg).cuda(), torch.from_numpy(conf).cuda(),
                         HN.to_device(x), y)


def test_copy_enqueue_failure_rolls_back():
    w = W2
    P = w.n_layers * w.n_experts
    raw = W.expert_blocks(w, 0, range(P))
    pool = HN.fill_pool(w, 0, P, raw=raw)
    ctx = HN.make_context(w, pool, copy_mode="sdma")
    ow = OracleWeights(w, 0, P, w.n_layers, raw=raw)
    lock = LockstepOracle(w.n_layers, w.n_experts, w.top_k, w.capacity)
    T, dt = w.tokens, HN.torch_dtype(w)
    y = torch.empty((T, w.hidden), dtype=dt, device="cuda")
    s = torch.cuda.current_stream()
    try:
        for l in range(w.n_layers):                      # iteration 0 fills both caches
            _step(ctx, w, l, 0, y)
            lg, conf, _ = _inputs(w, l, 0)
            lock.step(l, lg, conf, ctx.read_layer_state(l, T), f"l={l} i=0")
        before = ctx.read_layer_state(0, T)
        _say(f"[failure] layer 0 resident {int(before['resident_after'].sum())}")
        # iteration 1, layer 0: its second miss copy cannot be enqueued
        lg, conf, x = _inputs(w, 0, 1)
        o = O.layer_step(lg, conf, lock.res[0], w.top_k, w.capacity)
        assert o["n_misses"] >= 1, "the failing layer-iteration must have misses"
        ctx.set_fault_injection(copy_fail_at=2)
        ctx.route_block(0, torch.from_numpy(lg).cuda(), T, s)
        ctx.moe_forward_cached(0, HN.to_device(x), y, s)
        st = oled.apply_misses(ctx.ctx, 0, None, None)
        assert st == oled.OLED_ERR_HIP
        assert "could not be enqueued" in oled.last_error(ctx.ctx)
        # the layer is idle again: its retention is not called
        assert oled.score_and_retain(ctx.ctx, 0, torch.from_numpy(conf).cuda(), s) == \
            oled.OLED_ERR_STATE
        after = ctx.read_layer_state(0, T)        # also checks slot conservation
        np.testing.assert_array_equal(after["resident_after"], before["resident_after"])
        np.testing.assert_array_equal(after["retained"], before["resident_after"])
        np.testing.assert_array_equal(after["slot_of"], before["slot_of"])
        np.testing.assert_array_equal(after["retain_key"], before["retain_key"])
        # the context goes on; the oracle skips the failed layer-iteration
        for it in (1, 2, 3):
            for l in range(w.n_layers):
                if (l, it) == (0, 1):
                    continue
                _step(ctx, w, l, it, y)
                lg, conf, x = _inputs(w, l, it)
                o = lock.step(l, lg, conf, ctx.read_layer_state(l, T), f"l={l} i={it}")
                y_ref = O.moe_output(O.decode(x), o["idx"], o["gates"], ow.fn(l))
                err = rel_l2(O.decode(HN.from_device(y)), y_ref)
                assert err <= tol(w), f"l={l} i={it}: rel L2 {err:.3e}"
        _say("[failure] copy enqueue failure rolled back; later iterations match the oracle")
    finally:
        ctx.close()
        pool.free()


def test_wait_deadline_then_reset():
    w = W2.replace(n_layers=1, capacity=26)
    P = w.n_experts + 1
    pool = HN.fill_pool(w, 0, P)
    ctx = HN.make_context(w, pool, copy_mode="sdma")
    T, dt = w.tokens, HN.torch_dtype(w)
    y = torch.empty((T, w.hidden), dtype=dt, device="cuda")
    s = torch.cuda.current_stream()
    try:
        # a cold iteration copies every active expert (about 264 MiB, several
        # ms over PCIe); the host gives up on the copies after 1 ms
        ctx.set_fault_injection(wait_deadline_ms=1)
        lg, conf, x = _inputs(w, 0, 0)
        ctx.route_block(0, torch.from_numpy(lg).cuda(), T, s)
        ctx.moe_forward_cached(0, HN.to_device(x), y, s)
        assert oled.apply_misses(ctx.ctx, 0, None, None) == oled.OLED_ERR_HIP
        assert "within 1 ms" in oled.last_error(ctx.ctx)
        assert oled.route_block(ctx.ctx, 0, torch.from_numpy(lg).cuda(), T, s) == \
            oled.OLED_ERR_STATE
        ctx.reset_cache()                          # waits for the device, empties the caches
        ctx.set_fault_injection()                  # default deadline
        _step(ctx, w, 0, 0, y)
        st = ctx.read_layer_state(0, T)
        o = O.layer_step(lg, conf, np.zeros(w.n_experts, bool), w.top_k, w.capacity)
        compare_control(st, o, T, "after reset", lg, conf, w.capacity)
        ow = OracleWeights(w, 0, P, 1)
        y_ref = O.moe_output(O.decode(x), o["idx"], o["gates"], ow.fn(0))
        err = rel_l2(O.decode(HN.from_device(y)), y_ref)
        assert err <= tol(w), f"rel L2 {err:.3e}"
        _say("[failure] deadline reported; reset context matches the oracle")
    finally:
        ctx.close()
        pool.free()


def test_fault_injection_arguments():
    w = W.WORKLOADS[1]
    pool = HN.fill_pool(w, 0, 8)
    ctx = HN.make_context(w, pool)
    try:
        lib = oled.load()
        assert lib.oled_set_fault_injection(None, 0, 0) == oled.OLED_ERR_INVALID_ARG
        assert lib.oled_set_fault_injection(ctx.ctx, -1, 0) == oled.OLED_ERR_INVALID_ARG
        assert lib.oled_set_fault_injection(ctx.ctx, 0, -5) == oled.OLED_ERR_INVALID_ARG
        assert lib.oled_set_fault_injection(ctx.ctx, 3, 100) == oled.OLED_OK
    finally:
        ctx.close()
        pool.free()
