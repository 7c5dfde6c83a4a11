"""oled_route_noalloc (no context, no allocation: its scratch is a file-scope
device array) against route_block on the same logits: top-k ids, gates,
histogram, offsets and permutation bit for bit, on two calls in a row with
the second block smaller, over every routing path (fused launch; one
wavefront per token with a one-workgroup permutation; one token per lane
with the chunked permutation); then the non-finite flag."""
import sys

import numpy as np
import pytest
import torch

from oracle import oled_oracle as O
from paper_2609_33385_amd import harness as HN
from paper_2609_33385_amd import oled
from paper_2609_33385_amd import workload as W

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    oled.load()


def _logits(T, E, seed):
    rng = np.random.default_rng(seed)
    z = rng.standard_normal(((T + 31) // 32, E)) * 3.0   # a preference per 32 tokens
    lg = np.repeat(z, 32, axis=0)[:T] + rng.standard_normal((T, E))
    lg = np.round(lg * 8) / 8            # a coarse grid: many exact ties
    return lg.astype(np.float32)


def _noalloc(lg_dev, T, E, k, s):
    dev = dict(topk_idx=torch.full((T * k,), -7, dtype=torch.int32, device="cuda"),
               gates=torch.full((T * k,), -1.0, dtype=torch.float32, device="cuda"),
               counts=torch.full((E,), -7, dtype=torch.int32, device="cuda"),
               offsets=torch.full((E + 1,), -7, dtype=torch.int32, device="cuda"),
               perm=torch.full((T * k,), -7, dtype=torch.int32, device="cuda"),
               inv_perm=torch.full((T * k,), -7, dtype=torch.int32, device="cuda"),
               nonfinite=torch.full((1,), 5, dtype=torch.int32, device="cuda"))
    st = oled.oled_route_noalloc(lg_dev, T, E, k, dev["topk_idx"], dev["gates"], dev["counts"],
                                 dev["offsets"], dev["perm"], dev["inv_perm"], dev["nonfinite"], s)
    assert st == oled.OLED_OK, oled.last_error(None)
    torch.cuda.synchronize()
    return {key: v.cpu().numpy() for key, v in dev.items()}


def _route_block(ctx, lg_dev, T, conf, s):
    ctx.route_block(0, lg_dev, T, s)
    ctx.apply_misses(0, report=False)
    ctx.score_and_retain(0, conf, s)
    return ctx.read_layer_state(0, T)


SEQUENCES = [  # (E, k, [T of each call]): the second call's block is smaller
    (128, 8, [65535, 3000]),   # one token per lane, chunked permutation
    (128, 8, [900, 100]),      # one wavefront per token + one-workgroup permutation, then fused
    (64, 6, [5000, 1000]),     # chunked, then wavefront per token
    (200, 3, [2049, 300]),     # chunked over 200 experts, then fused
    (8, 2, [37, 5]),           # fused, small
]


@pytest.mark.parametrize("E,k,Ts", SEQUENCES)
def test_noalloc_matches_route_block(E, k, Ts):
    _say(f"[noalloc] E={E} k={k} T={Ts}")
    w = W.WORKLOADS[1].replace(wid=400, name="noalloc", dtype="bf16", batch=1, block=max(Ts),
                               n_experts=E, top_k=k, hidden=128, inter=128, n_layers=1,
                               n_iters=1, capacity=E // 3)
    pool = HN.fill_pool(w, 0, 2)
    ctx = HN.make_context(w, pool, max_tokens=max(Ts))
    s = torch.cuda.current_stream()
    try:
        for n, T in enumerate(Ts):
            lg = _logits(T, E, 1000 * E + n)
            lg_dev = torch.from_numpy(lg).cuda()
            got = _noalloc(lg_dev, T, E, k, s)
            conf = torch.full((T,), 0.5, dtype=torch.float32, device="cuda")
            ref = _route_block(ctx, lg_dev, T, conf, s)
            where = f"E={E} k={k} T={T} (call {n})"
            np.testing.assert_array_equal(got["topk_idx"].reshape(T, k), ref["topk_idx"],
                                          err_msg=where)
            np.testing.assert_array_equal(got["gates"].view(np.uint32),
                                          ref["gates"].reshape(-1).view(np.uint32), err_msg=where)
            for key in ("counts", "offsets", "perm", "inv_perm"):
                np.testing.assert_array_equal(got[key], ref[key], err_msg=f"{where} {key}")
            assert got["nonfinite"][0] == 0, where
            if T <= 5000:   # the integer results also against the oracle's permutation
                counts, offsets, perm, inv = O.permute(got["topk_idx"].reshape(T, k), E)
                np.testing.assert_array_equal(got["perm"], perm, err_msg=where)
                np.testing.assert_array_equal(got["offsets"], offsets, err_msg=where)
        _say("[noalloc] ok")
    finally:
        ctx.close()
        pool.free()


@pytest.mark.parametrize("E,k,T", [(16, 4, 40), (64, 8, 3000)])
def test_noalloc_nonfinite_flag(E, k, T):
    """A NaN or infinite logit sets the flag; the next good call clears it."""
    s = torch.cuda.current_stream()
    lg = _logits(T, E, 7)
    bad = lg.copy()
    bad[T // 2, 1] = np.nan if T < 100 else np.inf
    got = _noalloc(torch.from_numpy(bad).cuda(), T, E, k, s)
    assert got["nonfinite"][0] == 1
    got = _noalloc(torch.from_numpy(lg).cuda(), T, E, k, s)
    assert got["nonfinite"][0] == 0
    idx, gates = O.route(lg, k)
    np.testing.assert_array_equal(got["topk_idx"].reshape(T, k), idx)
