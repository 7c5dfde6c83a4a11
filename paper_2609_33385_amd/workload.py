"""Seeded synthetic inputs for the block-MoE layer under partial expert residency.

This module only draws numbers. It holds none of the method's arithmetic: no
routing, no softmax, no FFN, no scoring. Both the HIP path (through the
binding) and the CPU oracle consume the arrays it returns, so the two sides
see identical input bits.

The paper's workloads (LLaDA2.0 models on GSM8K / HumanEval / GPQA, Sec. 5.1)
need trained weights and datasets; these generators stand in for them with the
shapes of each workload and the statistics the paper states in prose:
a block of tokens refined over several denoising iterations (Sec. 2.1), roughly
a quarter to a third of the experts active per layer (Sec. 5.2), and high
overlap of the active expert set between adjacent iterations (Sec. 3.3).

Random-number scheme: every tensor is drawn from numpy's PCG64 seeded by
``SeedSequence(seed, spawn_key=(workload_id, tensor_id, layer, block, iter))``.
Values are drawn in float64 and emitted as float32 (logits, confidence) or
rounded to the workload dtype (activations, weights). bf16 values are carried
as uint16 bit patterns, rounded to nearest-even through float32.
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

# tensor ids inside the spawn key
_TID_PREF = 1     # per-sequence expert preference z[b][e]
_TID_NOISE = 2    # per-token logit noise n[t][e] at the first iteration of a block
_TID_STEP = 3     # iteration-to-iteration logit steps eps[i][t][e]
_TID_ZIPF = 4     # per-layer popularity rank permutation
_TID_CONF = 5     # confidence draws
_TID_X = 6        # activations
_TID_W = 7        # expert weight blocks
_TID_GATE = 8     # gate weights


@dataclasses.dataclass(frozen=True)
class Workload:
    """Shape and statistics of one synthetic workload."""

    wid: int              # workload id, part of every seed key
    name: str
    dtype: str            # "f32" or "bf16": dtype of activations, weights, outputs
    batch: int            # sequences per iteration
    block: int            # tokens per sequence block
    n_experts: int
    top_k: int
    hidden: int
    inter: int            # expert SwiGLU intermediate size
    n_layers: int
    n_iters: int          # denoising iterations per block
    capacity: int         # expert-cache slots per layer
    sigma_s: float = 3.0  # weight of the per-sequence expert preference
    sigma_it: float = 0.3 # std of the logit step between adjacent iterations
    zipf_s: float = 0.0   # >0: per-layer Zipf(s) popularity bias on logits
    conf_kind: str = "unmask"   # "beta22" | "uniform" | "unmask"
    sigma_s_layers: tuple = ()  # non-empty: sigma_s of layer l is sigma_s_layers[l % len]
    conf_informed: bool = False # steps of token t scaled by 2 (1 - its previous confidence)

    @property
    def tokens(self) -> int:
        return self.batch * self.block

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2

    @property
    def expert_elems(self) -> int:
        """Elements in one expert block: w13 [2I][H] followed by w2 [H][I]."""
        return 3 * self.hidden * self.inter

    @property
    def expert_bytes(self) -> int:
        return self.expert_elems * self.elem_bytes

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


def _cap(frac: float, n_experts: int) -> int:
    """Capacity for a residency fraction: round half up of frac * E."""
    return int(math.floor(frac * n_experts + 0.5))


# The five workloads. Shapes follow the LLaDA-MoE-like layer stacks used for
# the hot path; residency 40% (20% for the stress case).
WORKLOADS = {
    1: Workload(1, "tiny-f32", "f32", 1, 32, 8, 2, 256, 512, 1, 4, 4,
                conf_kind="beta22"),
    2: Workload(2, "llada-moe-b1", "bf16", 1, 32, 64, 8, 2048, 1024, 16, 8,
                _cap(0.4, 64)),
    3: Workload(3, "llada-moe-b8", "bf16", 8, 32, 64, 8, 2048, 1024, 16, 8,
                _cap(0.4, 64)),
    4: Workload(4, "e128-zipf-b16", "bf16", 16, 64, 128, 8, 4096, 1536, 48, 16,
                _cap(0.4, 128), zipf_s=1.1),
    5: Workload(5, "e128-stress-b16", "bf16", 16, 64, 128, 8, 4096, 1536, 48, 16,
                _cap(0.2, 128), sigma_it=1.5, conf_kind="uniform"),
}


def _rng(w: Workload, seed: int, tid: int, layer: int = 0, blk: int = 0,
         it: int = 0) -> np.random.Generator:
    ss = np.random.SeedSequence(seed, spawn_key=(w.wid, tid, layer, blk, it))
    return np.random.Generator(np.random.PCG64(ss))


# ---------------------------------------------------------------- encodings
def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16, nearest-even; returns uint16 bit patterns."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    rounding = np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return ((u + rounding) >> np.uint32(16)).astype(np.uint16)


def _emit(w: Workload, v64: np.ndarray) -> np.ndarray:
    v32 = v64.astype(np.float32)
    return v32 if w.dtype == "f32" else f32_to_bf16_bits(v32)


# ------------------------------------------------------------------- logits
def _layer_bias(w: Workload, seed: int, layer: int) -> np.ndarray:
    """Zipf(s) popularity bias: -s * ln(rank), rank a seeded permutation of 1..E."""
    if w.zipf_s <= 0.0:
        return np.zeros(w.n_experts)
    rank = _rng(w, seed, _TID_ZIPF, layer).permutation(w.n_experts) + 1
    return -w.zipf_s * np.log(rank.astype(np.float64))


def logits_block(w: Workload, seed: int, layer: int, blk: int) -> np.ndarray:
    """Router logits of one layer for every iteration of one block: float32 [N][T][E].

    Iteration 0 is sigma_s * z[seq] + n + bias (sigma_s per layer if
    sigma_s_layers is set: layers that route with different spread); each later
    iteration adds an independent N(0, sigma_it^2) step (a random walk, so
    adjacent iterations route mostly to the same experts). With conf_informed
    the step of token t at iteration i is scaled by 2 (1 - c_t^{i-1}), so the
    routes of confident tokens persist, as the paper observes of real
    denoising (Sec. 4.3).
    """
    T, E, N = w.tokens, w.n_experts, w.n_iters
    z = _rng(w, seed, _TID_PREF, layer).standard_normal((w.batch, E))
    n = _rng(w, seed, _TID_NOISE, layer, blk).standard_normal((T, E))
    sig = w.sigma_s_layers[layer % len(w.sigma_s_layers)] if w.sigma_s_layers else w.sigma_s
    base = sig * np.repeat(z, w.block, axis=0) + n + _layer_bias(w, seed, layer)
    steps = _rng(w, seed, _TID_STEP, layer, blk).standard_normal((N, T, E))
    steps[0] = 0.0
    if w.conf_informed:   # confident tokens move less: their routes persist (Sec. 4.3)
        for i in range(1, N):
            c = confidence(w, seed, blk, i - 1).astype(np.float64)
            steps[i] *= 2.0 * (1.0 - c)[:, None]
    walk = np.cumsum(w.sigma_it * steps, axis=0)
    return (base[None] + walk).astype(np.float32)


def logits(w: Workload, seed: int, layer: int, blk: int, it: int) -> np.ndarray:
    """Router logits float32 [T][E] of (layer, block, iteration)."""
    return logits_block(w, seed, layer, blk)[it]


# --------------------------------------------------------------- confidence
def confidence(w: Workload, seed: int, blk: int, it: int) -> np.ndarray:
    """Token confidence float32 [T] at (block, iteration), shared by all layers.

    "unmask": each sequence's block is split into n_iters equal groups by a
    seeded permutation; a token of group u has confidence
    c0 + (1 - c0) * min(1, (it + 1) / (u + 1)) with c0 ~ U(0, 0.5), rising
    monotonically and reaching 1 at the iteration it is unmasked.
    """
    T = w.tokens
    if w.conf_kind == "beta22":
        return _rng(w, seed, _TID_CONF, 0, blk, it).beta(2.0, 2.0, T).astype(np.float32)
    if w.conf_kind == "uniform":
        return _rng(w, seed, _TID_CONF, 0, blk, it).uniform(0.0, 1.0, T).astype(np.float32)
    r = _rng(w, seed, _TID_CONF, 0, blk)
    c0 = r.uniform(0.0, 0.5, T)
    group = max(1, w.block // w.n_iters)
    u = np.empty(T, dtype=np.int64)
    for b in range(w.batch):
        pos = r.permutation(w.block)
        u[b * w.block + pos] = np.minimum(np.arange(w.block) // group, w.n_iters - 1)
    c = c0 + (1.0 - c0) * np.minimum(1.0, (it + 1.0) / (u + 1.0))
    return np.clip(c, 0.0, 1.0).astype(np.float32)


# -------------------------------------------------------------- activations
def activations(w: Workload, seed: int, layer: int, blk: int, it: int) -> np.ndarray:
    """Layer input [T][H] ~ N(0, 0.02^2): float32, or uint16 bf16 bits."""
    v = 0.02 * _rng(w, seed, _TID_X, layer, blk, it).standard_normal((w.tokens, w.hidden))
    return _emit(w, v)


# ------------------------------------------------------------------ weights
def expert_block(w: Workload, seed: int, b: int) -> np.ndarray:
    """Host weight block b, flat [3*H*I] in the workload dtype encoding.

    Layout: w13 [2I][H] row-major (gate projection rows, then up projection
    rows) followed by w2 [H][I] row-major. Entries ~ N(0, 0.02^2).
    """
    r = _rng(w, seed, _TID_W, 0, b)
    v = 0.02 * r.standard_normal(w.expert_elems)
    return _emit(w, v)


def expert_blocks(w: Workload, seed: int, blocks, threads: int = 16) -> dict:
    """{b: expert_block(w, seed, b)} for the given block ids, drawn on a thread
    pool (the draws and conversions release the GIL). Same bits as drawing
    them one by one."""
    import concurrent.futures
    ids = [int(b) for b in blocks]
    with concurrent.futures.ThreadPoolExecutor(max(1, threads)) as ex:
        return dict(zip(ids, ex.map(lambda b: expert_block(w, seed, b), ids)))


def gate_weights(w: Workload, seed: int, layer: int) -> np.ndarray:
    """Gate weights of a layer [E][H] in the workload dtype encoding, entries
    ~ N(0, (150 / sqrt(H))^2), so that logits of N(0, 0.02^2) activations have
    a standard deviation of about 3."""
    r = _rng(w, seed, _TID_GATE, layer)
    v = (150.0 / math.sqrt(w.hidden)) * r.standard_normal((w.n_experts, w.hidden))
    return _emit(w, v)


def host_block_of(w: Workload, n_blocks: int) -> np.ndarray:
    """Expert (layer l, expert e) -> host block (l*E + e) mod P, int64 [L*E].

    With n_blocks < L*E several experts alias one host block; the transfer
    volume per miss is unchanged.
    """
    return (np.arange(w.n_layers * w.n_experts, dtype=np.int64) % n_blocks)


def split_expert(w: Workload, block: np.ndarray):
    """Views (w13 [2I][H], w2 [H][I]) of a flat expert block."""
    H, I = w.hidden, w.inter
    return block[: 2 * I * H].reshape(2 * I, H), block[2 * I * H:].reshape(H, I)
