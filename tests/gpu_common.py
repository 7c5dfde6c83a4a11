"""Shared helpers of the GPU parity tests: run a schedule through the C ABI and
through the oracle on the same seeded inputs, and compare."""
from __future__ import annotations

import numpy as np
import torch

from oracle import oled_oracle as O
from paper_2609_33385_amd import harness as HN
from paper_2609_33385_amd import workload as W


def rel_l2(a: np.ndarray, b: np.ndarray) -> float:
    d = np.linalg.norm(np.asarray(a, np.float64) - np.asarray(b, np.float64))
    n = np.linalg.norm(np.asarray(b, np.float64))
    return float(d / n) if n > 0 else float(d)


def tol(w: W.Workload) -> float:
    """Relative L2 bound on layer outputs: 1e-5 in fp32, 2e-2 in bf16."""
    return 1e-5 if w.dtype == "f32" else 2e-2


class OracleWeights:
    """float64 expert weights of a host pool, decoded once per block."""

    def __init__(self, w: W.Workload, seed: int, n_blocks: int, n_layers: int):
        self.w, self.seed, self.P = w, seed, n_blocks
        self.hbo = W.host_block_of(w.replace(n_layers=n_layers), n_blocks)
        self.cache = {}

    def block(self, b: int):
        if b not in self.cache:
            flat = O.decode(W.expert_block(self.w, self.seed, b))
            w13, w2 = W.split_expert(self.w, flat)
            self.cache[b] = (w13, w2)
        return self.cache[b]

    def fn(self, layer: int):
        E = self.w.n_experts
        return lambda e: self.block(int(self.hbo[layer * E + e]))


def compare_control(st_gpu: dict, st_or: dict, T: int, where: str):
    assert st_gpu["tokens"] == T, where
    np.testing.assert_array_equal(st_gpu["topk_idx"], st_or["idx"], err_msg=where + " idx")
    np.testing.assert_array_equal(st_gpu["gates"].view(np.uint32),
                                  st_or["gates"].view(np.uint32), err_msg=where + " gates")
    np.testing.assert_array_equal(st_gpu["counts"], st_or["counts"], err_msg=where + " counts")
    np.testing.assert_array_equal(st_gpu["offsets"], st_or["offsets"], err_msg=where + " offsets")
    np.testing.assert_array_equal(st_gpu["perm"], st_or["perm"], err_msg=where + " perm")
    np.testing.assert_array_equal(st_gpu["inv_perm"], st_or["inv_perm"], err_msg=where + " inv_perm")
    assert st_gpu["n_active"] == st_or["n_active"], where
    assert st_gpu["n_hits"] == st_or["n_hits"], where
    assert st_gpu["n_misses"] == st_or["n_misses"], where
    np.testing.assert_array_equal(st_gpu["resident_before"], st_or["resident_before"],
                                  err_msg=where + " R before")
    np.testing.assert_array_equal(st_gpu["score_q"], st_or["S"], err_msg=where + " scores")
    np.testing.assert_array_equal(st_gpu["resident_after"], st_or["resident_after"],
                                  err_msg=where + " R after")


def run_schedule_gpu(ctx, w: W.Workload, seed: int, layers, n_iters: int, forward: bool,
                     on_step=None, report: bool = True):
    """Runs iterations 0..n_iters-1 of block 0 over the given workload layers.

    Context layer li stands for workload layer layers[li]. on_step(i, li, state,
    y, rep) is called after each layer-iteration (state from
    oled_read_layer_state, rep the miss report or None).
    """
    dt = HN.torch_dtype(w)
    T = w.tokens
    for i in range(n_iters):
        conf = torch.from_numpy(W.confidence(w, seed, 0, i)).cuda()
        for li, l in enumerate(layers):
            logits = torch.from_numpy(W.logits(w, seed, l, 0, i)).cuda()
            x = y = None
            if forward:
                x = HN.to_device(W.activations(w, seed, l, 0, i))
                y = torch.empty((T, w.hidden), dtype=dt, device="cuda")
            rep = HN.layer_step(ctx, li, logits, conf, x, y, report=report)
            state = ctx.read_layer_state(li, T)
            if on_step is not None:
                on_step(i, li, state, None if y is None else HN.from_device(y), rep)


def check_report(rep, st_or: dict, eb: int, where: str):
    """A miss report against the oracle's layer step (every miss is transferred)."""
    if rep is None:
        return
    assert (rep.n_active, rep.n_hits, rep.n_misses) == (
        st_or["n_active"], st_or["n_hits"], st_or["n_misses"]), where
    assert rep.n_resident == int(np.count_nonzero(st_or["resident_before"])), where
    assert rep.h2d_bytes == st_or["n_misses"] * eb, where


def oracle_schedule(w: W.Workload, seed: int, layers, n_iters: int, capacity: int):
    return O.run_schedule(lambda li, i: W.logits(w, seed, layers[li], 0, i),
                          lambda li, i: W.confidence(w, seed, 0, i),
                          len(layers), n_iters, w.n_experts, w.top_k, capacity)
