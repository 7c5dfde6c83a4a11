"""Drives the block-MoE layer stack of a synthetic workload through the C ABI.

Used by the GPU tests, the smoke check and the benchmark. Every step of the
hot path runs in liboled.so; this module prepares seeded inputs (workload.py),
fills the pinned host expert pool, moves inputs to the device with PyTorch and
issues the four ABI calls per layer.
"""
from __future__ import annotations

import numpy as np
import torch

from . import oled
from . import workload as W


def fill_pool(w: W.Workload, seed: int, n_blocks: int, raw: dict | None = None,
              threads: int = 16) -> oled.PinnedPool:
    """Pinned host pool of n_blocks expert blocks drawn by workload.expert_block
    (or taken from `raw`, {block: drawn block}), packed into the library's
    expert-block layout on a thread pool (the draws and the packing call
    release the GIL)."""
    import concurrent.futures
    pool = oled.PinnedPool(n_blocks, w.expert_bytes)
    dt = np.float32 if w.dtype == "f32" else np.uint16

    def one(b):
        flat = raw[b] if raw is not None else W.expert_block(w, seed, b)
        w13, w2 = W.split_expert(w, flat)
        oled.oled_pack_expert(w.dtype, w.hidden, w.inter, w13, w2, pool.block(b, dt))

    try:
        with concurrent.futures.ThreadPoolExecutor(max(1, min(threads, n_blocks))) as ex:
            list(ex.map(one, range(n_blocks)))
    except BaseException:
        pool.free()
        raise
    return pool


def make_context(w: W.Workload, pool: oled.PinnedPool, capacity: int | None = None,
                 n_layers: int | None = None, max_tokens: int | None = None,
                 profile_ops: int = 0, copy_mode: str = "shader",
                 adapt_period: int = 0, policy: str = "priority",
                 coop: dict | None = None) -> oled.Context:
    L = n_layers if n_layers is not None else w.n_layers
    return oled.Context(w.hidden, w.inter, w.n_experts, w.top_k, L,
                        w.capacity if capacity is None else capacity,
                        max_tokens if max_tokens is not None else w.tokens, w.dtype,
                        pool.ptr, pool.n_blocks,
                        W.host_block_of(w.replace(n_layers=L), pool.n_blocks), profile_ops=profile_ops,
                        copy_mode=copy_mode, adapt_period=adapt_period, policy=policy, coop=coop)


def torch_dtype(w: W.Workload):
    return torch.float32 if w.dtype == "f32" else torch.bfloat16


def to_device(a: np.ndarray, dtype=None, device="cuda") -> torch.Tensor:
    """Host array -> device tensor with the same bits (uint16 arrays become bf16)."""
    if a.dtype == np.uint16:
        t = torch.from_numpy(a.view(np.int16).copy()).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(a))
    return t.to(device)


def from_device(t: torch.Tensor) -> np.ndarray:
    """Device tensor -> host array with the same bits (bf16 becomes uint16)."""
    t = t.detach().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def layer_step(ctx: oled.Context, layer: int, logits: torch.Tensor, conf: torch.Tensor,
               x: torch.Tensor | None = None, y: torch.Tensor | None = None,
               stream=None, report: bool = True) -> oled.MissReport | None:
    """route_block -> [moe_forward_cached] -> apply_misses -> score_and_retain."""
    s = stream if stream is not None else torch.cuda.current_stream()
    T = logits.shape[0]
    ctx.route_block(layer, logits, T, s)
    if x is not None:
        ctx.moe_forward_cached(layer, x, y, s)
    if getattr(ctx, "coop", False):
        rep = ctx.apply_misses_coop(layer, conf, report=report)
    else:
        rep = ctx.apply_misses(layer, report=report)
    ctx.score_and_retain(layer, conf, s)
    return rep
