"""GPU parity of the comparison retention policies (LRU, LFU; Sec. 5.1 and
Sec. 5.3) and of the effective-transfer counters against the oracle: the
control path bit for bit at every layer-iteration (the retention key of every
expert included), the routing totals, and layer outputs that do not depend on
the policy (bitwise equal to the priority policy's)."""
import sys

import numpy as np
import pytest
import torch

from oracle import oled_oracle as O
from paper_2609_33385_amd import harness as HN
from paper_2609_33385_amd import oled
from paper_2609_33385_amd import workload as W

from gpu_common import compare_control, run_schedule_gpu

pytestmark = pytest.mark.gpu

STACK = W.WORKLOADS[2].replace(wid=330, name="policy-stack", n_layers=4, n_iters=8, capacity=16)


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    oled.load()


def _oracle(w, seed, C, policy, period=0):
    return O.run_schedule(lambda li, i: W.logits(w, seed, li, 0, i),
                          lambda li, i: W.confidence(w, seed, 0, i),
                          w.n_layers, w.n_iters, w.n_experts, w.top_k, C, policy=policy,
                          adapt_period=period)


def _chain(w, seed, C, policy, period=0, forward=False, outs=None):
    L = w.n_layers
    _say(f"[policy] {w.name} policy={policy} C={C} period={period} forward={forward}")
    ref = _oracle(w, seed, C, policy, period)
    pool = HN.fill_pool(w, seed, w.n_experts + 1)
    ctx = HN.make_context(w, pool, capacity=C, policy=policy, adapt_period=period)

    def check(i, li, st, y, rep):
        o = ref[i][li]
        where = f"{policy} l={li} i={i}"
        resized = li == L - 1 and "capacities_after" in o
        if resized:
            for lj in range(L):
                sj = ctx.read_layer_state(lj, w.tokens)
                np.testing.assert_array_equal(sj["resident_after"], o["residents_after_update"][lj],
                                              err_msg=f"{where} layer {lj} after re-sizing")
        compare_control(st, o, w.tokens, where, W.logits(w, seed, li, 0, i),
                        W.confidence(w, seed, 0, i), o["capacity"], policy=policy,
                        state_after=o["residents_after_update"][li] if resized else None)
        np.testing.assert_array_equal(st["retain_key"], o["key"], err_msg=where + " key")
        assert (st["prev_transferred"], st["reused_transfers"]) == (
            o["prev_transferred"], o["reused_transfers"]), where
        if outs is not None and y is not None:
            outs.append(y.copy())

    try:
        ctx.collect_stats()
        run_schedule_gpu(ctx, w, seed, list(range(L)), w.n_iters, forward, check)
        stats = ctx.collect_stats()
    finally:
        ctx.close()
        pool.free()
    flat = [o for row in ref for o in row]
    assert stats["n_prev_transferred"] == sum(o["prev_transferred"] for o in flat)
    assert stats["n_transfers_reused"] == sum(o["reused_transfers"] for o in flat)
    if period == 0:
        assert stats["n_ideal_hits"] == sum(O.ideal_hits(o["n_active"], C) for o in flat)
    _say(f"[policy] ok: hits {sum(o['n_hits'] for o in flat)}, effective transfer ratio "
         f"{O.effective_transfer_ratio(ref):.3f}")


@pytest.mark.parametrize("policy", ["priority", "lru", "lfu"])
@pytest.mark.parametrize("C", [6, 16])
def test_policy_control_path(policy, C):
    _chain(STACK, 0, C, policy)


def test_policy_with_adaptive_sizing():
    w = STACK.replace(sigma_s_layers=(0.5, 2.0, 3.5, 6.0))
    _chain(w, 1, 16, "lru", period=2)


def test_outputs_do_not_depend_on_policy():
    w = STACK.replace(n_iters=4)
    outs = {}
    for policy in ("priority", "lru", "lfu"):
        outs[policy] = []
        _chain(w, 2, 10, policy, forward=True, outs=outs[policy])
    for policy in ("lru", "lfu"):
        for a, b in zip(outs["priority"], outs[policy]):
            assert np.array_equal(a, b), policy
