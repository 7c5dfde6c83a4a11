"""GPU parity of the batched, context-free routing and priority calls
(oled_route_batch, oled_priority_batch) over B independent blocks: every
block's top-k ids, counts, offsets and permutation bit for bit against the
oracle (gates bit for bit up to the one-ulp float64-exp rule of the other
GPU tests), and bit for bit against route_block on the same block; priority
numerators exactly against the oracle; per-block non-finite and confidence
flags."""
import sys

import numpy as np
import pytest
import torch

from oracle import oled_oracle as O
from paper_2609_33385_amd import harness as HN
from paper_2609_33385_amd import oled
from paper_2609_33385_amd import workload as W

from gpu_common import accepted_gate_flip

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    oled.load()


def _logits(B, T, E, seed):
    rng = np.random.default_rng(seed)
    z = rng.standard_normal((B, (T + 63) // 64, E)) * 3.0
    lg = np.repeat(z, 64, axis=1)[:, :T] + rng.standard_normal((B, T, E))
    lg[:, ::7] = np.round(lg[:, ::7] * 4) / 4     # exact ties on some tokens
    return lg.astype(np.float32)


def _route_batch(lg, k):
    B, T, E = lg.shape
    s = torch.cuda.current_stream()
    dev = dict(topk_idx=torch.full((B, T * k), -7, dtype=torch.int32, device="cuda"),
               gates=torch.full((B, T * k), -1.0, dtype=torch.float32, device="cuda"),
               counts=torch.full((B, E), -7, dtype=torch.int32, device="cuda"),
               offsets=torch.full((B, E + 1), -7, dtype=torch.int32, device="cuda"),
               perm=torch.full((B, T * k), -7, dtype=torch.int32, device="cuda"),
               inv_perm=torch.full((B, T * k), -7, dtype=torch.int32, device="cuda"),
               nonfinite=torch.full((B,), 9, dtype=torch.int32, device="cuda"))
    ws = torch.empty(oled.oled_route_batch_workspace(B, T, E), dtype=torch.uint8, device="cuda")
    st = oled.oled_route_batch(torch.from_numpy(lg).cuda(), B, T, E, k, dev["topk_idx"],
                               dev["gates"], dev["counts"], dev["offsets"], dev["perm"],
                               dev["inv_perm"], dev["nonfinite"], ws, s)
    assert st == oled.OLED_OK, oled.last_error(None)
    torch.cuda.synchronize()
    return {key: v.cpu().numpy() for key, v in dev.items()}


def _check_block(got, b, lg_b, k, where):
    T, E = lg_b.shape
    idx, gates = O.route(lg_b, k)
    np.testing.assert_array_equal(got["topk_idx"][b].reshape(T, k), idx, err_msg=where)
    g = got["gates"][b].reshape(T, k)
    for t, j in np.argwhere(g.view(np.uint32) != gates.view(np.uint32)):
        assert accepted_gate_flip(lg_b[t], idx[t], j, g[t, j], gates[t, j]), (where, t, j)
    counts, offsets, perm, inv = O.permute(idx, E)
    for key, ref in (("counts", counts), ("offsets", offsets), ("perm", perm),
                     ("inv_perm", inv)):
        np.testing.assert_array_equal(got[key][b], ref, err_msg=f"{where} {key}")
    assert got["nonfinite"][b] == 0, where


@pytest.mark.parametrize("B,T,E,k", [(4, 3000, 128, 8), (3, 100, 200, 3), (5, 513, 64, 6),
                                     (2, 1, 8, 2),
                                     # streamed top-k (E a multiple of 32, k <= 8): one and
                                     # eight 32-expert chunks; register staging at k = 16
                                     # (E = 96) and at E = 48
                                     (2, 2500, 32, 4), (2, 1100, 96, 16), (2, 1500, 256, 8),
                                     (2, 1300, 48, 8)])
def test_route_batch_against_oracle(B, T, E, k):
    _say(f"[batch] route B={B} T={T} E={E} k={k}")
    lg = _logits(B, T, E, 10 * B + k)
    got = _route_batch(lg, k)
    for b in range(B):
        _check_block(got, b, lg[b], k, f"B={B} T={T} E={E} k={k} block {b}")


def test_route_batch_largest_blocks():
    """Two blocks of 65535 tokens: block 0 against the oracle, block 1 bit for
    bit against route_block."""
    B, T, E, k = 2, 65535, 128, 8
    lg = _logits(B, T, E, 77)
    got = _route_batch(lg, k)
    _check_block(got, 0, lg[0], k, "largest block 0")
    w = W.WORKLOADS[2].replace(wid=410, name="batch-ref", batch=1, block=T, n_experts=E,
                               top_k=k, hidden=128, inter=128, n_layers=1, n_iters=1,
                               capacity=E // 3)
    pool = HN.fill_pool(w, 0, 2)
    ctx = HN.make_context(w, pool)
    s = torch.cuda.current_stream()
    try:
        ctx.route_block(0, torch.from_numpy(lg[1]).cuda(), T, s)
        ctx.apply_misses(0, report=False)
        ctx.score_and_retain(0, torch.full((T,), 0.5, device="cuda"), s)
        ref = ctx.read_layer_state(0, T)
    finally:
        ctx.close()
        pool.free()
    np.testing.assert_array_equal(got["topk_idx"][1], ref["topk_idx"].reshape(-1))
    np.testing.assert_array_equal(got["gates"][1].view(np.uint32),
                                  ref["gates"].reshape(-1).view(np.uint32))
    for key in ("counts", "offsets", "perm", "inv_perm"):
        np.testing.assert_array_equal(got[key][1], ref[key], err_msg=key)


def test_route_batch_nonfinite_flags():
    B, T, E, k = 3, 1500, 64, 4
    lg = _logits(B, T, E, 5)
    lg[1, 777, 3] = np.nan
    got = _route_batch(lg, k)
    assert list(got["nonfinite"]) == [0, 1, 0]
    for b in (0, 2):
        _check_block(got, b, lg[b], k, f"block {b} beside a bad one")


def test_route_batch_unaligned_route_arrays():
    """topk_idx and inv_perm 4 bytes off a 16-byte boundary: at k = 8 the
    counting and ranking launches then take their 4-byte paths instead of the
    16-byte loads and stores; every output equals the aligned call's."""
    B, T, E, k = 2, 1500, 128, 8
    _say(f"[batch] unaligned route arrays B={B} T={T} E={E} k={k}")
    lg = _logits(B, T, E, 77)
    ref = _route_batch(lg, k)
    s = torch.cuda.current_stream()
    R = T * k
    raw = {name: torch.full((B * R + 1,), -7, dtype=torch.int32, device="cuda")
           for name in ("topk_idx", "inv_perm")}
    dev = dict(topk_idx=raw["topk_idx"][1:],
               gates=torch.full((B * R,), -1.0, dtype=torch.float32, device="cuda"),
               counts=torch.full((B * E,), -7, dtype=torch.int32, device="cuda"),
               offsets=torch.full((B * (E + 1),), -7, dtype=torch.int32, device="cuda"),
               perm=torch.full((B * R,), -7, dtype=torch.int32, device="cuda"),
               inv_perm=raw["inv_perm"][1:],
               nonfinite=torch.full((B,), 9, dtype=torch.int32, device="cuda"))
    assert dev["topk_idx"].data_ptr() % 16 == 4 and dev["inv_perm"].data_ptr() % 16 == 4
    ws = torch.empty(oled.oled_route_batch_workspace(B, T, E), dtype=torch.uint8, device="cuda")
    st = oled.oled_route_batch(torch.from_numpy(lg).cuda(), B, T, E, k, dev["topk_idx"],
                               dev["gates"], dev["counts"], dev["offsets"], dev["perm"],
                               dev["inv_perm"], dev["nonfinite"], ws, s)
    assert st == oled.OLED_OK, oled.last_error(None)
    torch.cuda.synchronize()
    got = {key: v.cpu().numpy() for key, v in dev.items()}
    for key in ("topk_idx", "counts", "offsets", "perm", "inv_perm", "nonfinite"):
        np.testing.assert_array_equal(got[key].reshape(-1), ref[key].reshape(-1), err_msg=key)
    np.testing.assert_array_equal(got["gates"].view(np.uint32),
                                  ref["gates"].reshape(-1).view(np.uint32))
    assert raw["topk_idx"][0].item() == -7 and raw["inv_perm"][0].item() == -7


@pytest.mark.parametrize("B,T,E,k", [(3, 3000, 128, 8), (2, 20000, 64, 8), (4, 37, 16, 4)])
def test_priority_batch_against_oracle(B, T, E, k):
    _say(f"[batch] priority B={B} T={T} E={E} k={k}")
    lg = _logits(B, T, E, 3 * T + k)
    got = _route_batch(lg, k)
    rng = np.random.default_rng(T)
    conf = rng.uniform(0, 1, (B, T)).astype(np.float32)
    conf[:, ::11] = 1.0
    conf[:, ::13] = 0.0
    s = torch.cuda.current_stream()
    S = torch.full((B, E), 123, dtype=torch.int64, device="cuda")
    bad = torch.full((B,), 9, dtype=torch.int32, device="cuda")
    topk = torch.from_numpy(got["topk_idx"]).cuda()
    gates = torch.from_numpy(got["gates"]).cuda()
    st = oled.oled_priority_batch(topk, gates, torch.from_numpy(conf).cuda(), B, T, E, k, S, bad, s)
    assert st == oled.OLED_OK, oled.last_error(None)
    torch.cuda.synchronize()
    S_gpu = S.cpu().numpy().view(np.uint64)
    assert list(bad.cpu().numpy()) == [0] * B
    for b in range(B):   # on the GPU's own routes and gates
        ref, _ = O.score(got["topk_idx"][b].reshape(T, k), got["gates"][b].reshape(T, k), conf[b], E)
        np.testing.assert_array_equal(S_gpu[b], ref, err_msg=f"block {b}")
    conf[B - 1, 5] = 1.5
    st = oled.oled_priority_batch(topk, gates, torch.from_numpy(conf).cuda(), B, T, E, k, S, bad, s)
    assert st == oled.OLED_OK
    torch.cuda.synchronize()
    assert list(bad.cpu().numpy()) == [0] * (B - 1) + [1]
