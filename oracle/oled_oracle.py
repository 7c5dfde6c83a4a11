"""CPU oracle of the block-MoE expert layer under partial expert residency.

TEST INFRASTRUCTURE ONLY. Only the tests, the smoke check of the build entry
point and the CPU-baseline leg of the benchmark may import this module. The
product path never calls it, and it shares no code with the HIP library.

What it computes, for one MoE layer l in one denoising iteration i of a
semi-autoregressive dLLM (OLED-MoE, Sec. 2.1 and Sec. 4), step by step and in
float64 from the exact input bits:

  O1 route      top-k experts per token and their gate scores (Sec. 2.1, 4.1)
  O2 permute    expert histogram, offsets, stable token permutation
  O3 classify   active set A, hits A & R, misses M = A \\ R (Sec. 4.2)
  O4 expert_ffn SwiGLU expert FFN
  O5 moe_output y[t] = sum_j g[t][j] * FFN_{idx[t][j]}(x[t]); it does not
                depend on R (the system is lossless, Sec. 5.1)
  O6 score      reuse-priority numerators (the priority equation of Sec. 4.3)
  O7            stale residents (resident, not activated) score zero (Sec. 4.3)
  O8 retain     R^{i+1} = Top_C(R^i u G^i, p) (the retention rule, Sec. 4.2),
                with G = M (every miss is transferred to the GPU)
  O9            R^{i+1} feeds the same layer at iteration i+1 (Sec. 4.1)
  O11 policies  the comparison retention policies of Sec. 5.1 / 5.3 (LRU,
                LFU) in place of the priority, the clairvoyant ideal cache
                bound, and the effective transfer ratio (Sec. 5.3)
  O13 gate      the gate's logits in front of O1 (Sec. 2.1): x W_gate^T in
                float64, and the bound on an fp32 accumulation of them
  O12 coop      cooperative compensation (Sec. 4.4): the hardware-aware
                split rho, and the two-stage load- and reuse-aware dispatch of
                the misses into transfers G and CPU executions M - G; only G
                joins the retention candidates
  O10 adapt     layer-adaptive cache sizing (Sec. 4.3): smoothed activation
                ratio a_l and cache utilisation u_l per layer, layer weight
                w_l = a_l * u_l and capacity C_l = C_total * w_l / sum_j w_j,
                recomputed every few iterations and enforced by evicting the
                lowest-priority residents of layers left over capacity

Readings where the paper is silent (each is restated in the design notes):
  * gate function: softmax over the k selected logits (equal to a full softmax
    renormalised over the top-k); exp and the sum in float64, sum in slot
    order, one round-to-nearest to float32;
  * ties in top-k: lower expert id first; slot order is (logit desc, id asc);
  * the gate score in the priority is the renormalised float32 gate;
  * psi(c) = c, the paper's default;
  * the priority numerator is accumulated exactly as integers,
    S[e] = sum floor(g * c * 2^48): g*c is exact in float64 (24+24 bits) and
    the floor is exact, so any summation order gives the same S. Ranking by S
    equals ranking by p_e because the denominator is one per-layer constant;
  * Top-C ties: (S desc, previously resident first, id asc); candidates with
    S = 0 are kept while capacity remains (eviction only when over capacity);
  * utilisation = hits / C (fraction of cache capacity serving activated
    experts, Sec. 3.2 and Sec. 5.1).
Readings of the comparison policies (O11), which the paper names but does not
define:
  * every policy keeps Top_C of the same candidates R u M and differs only in
    the primary key, with the same tie-breaks (previously resident first, id
    asc): LRU ranks by the layer iteration in which the expert was last
    activated (iterations of the layer counted from 1 since the empty cache);
    LFU by the number of routes (tokens) sent to it in the layer since the
    empty cache, evicted or not;
  * ideal cache bound: with perfect knowledge of A, the most activated experts
    a cache of C can hold before the layer runs, min(C, |A|) hits;
  * effective transfer ratio: of the experts transferred at a layer's
    iteration i, the share retained and activated again at its iteration
    i + 1, summed over iterations that have a next one.
Readings of the cooperative compensation (O12), where the paper names the
objective J(G) = T_comp - lambda * sum_{e in G} p_e and a two-stage heuristic
but not the cost model or the bounds:
  * T_comp(G) = max(T_H2D * |G|, tau_CPU * sum_{e in M - G} n_e): the transfer
    path and the CPU path run in parallel (n_e = routed tokens of e); the GPU
    compute of transferred experts is left out;
  * rho = nbar tau_CPU / (nbar tau_CPU + T_H2D); stage 1 transfers the
    round_half_up(rho |M|) misses of highest priority (S desc, id asc);
  * stage 2: at most |M| swaps of one transferred and one CPU expert, each the
    best swap by J (first in (transferred id, CPU id) order among equals),
    taken only if it lowers J strictly; swaps keep |G| at the hardware-aware
    split;
  * sum_{e in G} p_e = (sum_{e in G} S_e) / (sum_e S_e) (0 if no mass), and
    every term in float64 in the order written; lambda is an input (time per
    unit of priority mass);
  * only G joins the retention candidates R u G; CPU-executed experts leave
    no trace in the cache.
Readings of the layer-adaptive sizing (O10), where the paper gives the
formulas but not the smoothing, the rounding or the enforcement:
  * smoothing: an exponential moving average with weight 1/2 on the newest
    observation, per layer, in float64: x <- obs / 2 + x / 2, starting at the
    first observation; a_obs = |A_l| / E, u_obs = hits_l / C_l (skipped while
    the layer has capacity 0);
  * the update runs after every `period` completed iterations of the whole
    layer stack (period 5 in the paper), counted from the empty cache;
  * integer capacities: proportional shares q_l = C_avail * w_l / W (W the sum
    of w over the layers still open, in layer order), layers whose share
    exceeds E are set to E and the rest re-shared, then the largest-remainder
    method: floor(q_l) each, and the leftover units one each to the open
    layers below E in order of (q_l - floor(q_l) desc, layer asc). If every
    w_l is 0 the capacities stay as they are;
  * enforcement: a layer holding more experts than its new capacity evicts at
    once its residents of lowest priority, ranked by (its last retention key
    desc, id asc), the key being the priority numerator S under the paper's
    policy; a layer whose capacity grew fills it at its next retentions. So at
    no time do the layers hold more than C_total experts.
"""
from __future__ import annotations

import math

import numpy as np

SCORE_SHIFT = 48
SCORE_SCALE = float(2 ** SCORE_SHIFT)


# ------------------------------------------------------------ input decoding
def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """uint16 bf16 bit patterns -> float64 (exact)."""
    u32 = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u32.view(np.float32).astype(np.float64)


def decode(a: np.ndarray) -> np.ndarray:
    """Workload-encoded array (float32, or uint16 bf16 bits) -> float64."""
    if a.dtype == np.uint16:
        return bf16_bits_to_f64(a)
    return np.asarray(a, dtype=np.float32).astype(np.float64)


# ----------------------------------------------------------------- O1 route
def route(logits: np.ndarray, k: int):
    """O1. Top-k routing of every token of the block, with gate scores.

    logits: float32 [T][E]. Returns idx int32 [T][k] ordered by
    (logit desc, expert id asc) and gates float32 [T][k]:
      gate[t][j] = fl32( e_j / (e_0 + ... + e_{k-1}) ),
      e_j = exp(logit[t][idx[t][j]] - logit[t][idx[t][0]]) in float64.
    """
    logits = np.asarray(logits, dtype=np.float32)
    if not np.all(np.isfinite(logits)):
        raise ValueError("non-finite router logit")
    T, E = logits.shape
    if not 1 <= k <= E:
        raise ValueError("top_k out of range")
    # stable sort on -logit keeps lower ids first among equal logits
    order = np.argsort(-logits.astype(np.float64), axis=1, kind="stable")
    idx = order[:, :k].astype(np.int32)
    gates = np.empty((T, k), dtype=np.float32)
    for t in range(T):
        sel = [float(logits[t, e]) for e in idx[t]]
        ex = [math.exp(v - sel[0]) for v in sel]
        s = 0.0
        for v in ex:
            s += v
        for j in range(k):
            gates[t, j] = np.float32(ex[j] / s)
    return idx, gates


# --------------------------------------------------------------- O2 permute
def permute(idx: np.ndarray, n_experts: int):
    """O2. Expert histogram, exclusive offsets and stable counting-sort permutation.

    Route r = t*k + j goes to position offsets[e] + #{t' < t : e in idx[t']}.
    Returns counts [E], offsets [E+1], perm [T*k] (position -> route) and
    inv_perm [T*k] (route -> position), all int32.
    """
    flat = np.asarray(idx, dtype=np.int64).ravel()
    counts = np.zeros(n_experts, dtype=np.int64)
    for e in flat:
        counts[e] += 1
    offsets = np.zeros(n_experts + 1, dtype=np.int64)
    for e in range(n_experts):
        offsets[e + 1] = offsets[e] + counts[e]
    seen = np.zeros(n_experts, dtype=np.int64)
    inv_perm = np.empty(flat.size, dtype=np.int64)
    for r, e in enumerate(flat):
        inv_perm[r] = offsets[e] + seen[e]
        seen[e] += 1
    perm = np.empty(flat.size, dtype=np.int64)
    perm[inv_perm] = np.arange(flat.size)
    return (counts.astype(np.int32), offsets.astype(np.int32),
            perm.astype(np.int32), inv_perm.astype(np.int32))


# -------------------------------------------------------------- O3 classify
def classify(counts: np.ndarray, resident: np.ndarray):
    """O3. Active set A, hit mask A & R, miss mask M = A \\ R (Sec. 4.2)."""
    active = np.asarray(counts) > 0
    resident = np.asarray(resident, dtype=bool)
    return active, active & resident, active & ~resident


# ------------------------------------------------------------ O4/O5 outputs
def silu(z: np.ndarray) -> np.ndarray:
    return z / (1.0 + np.exp(-z))


def expert_ffn(x: np.ndarray, w13: np.ndarray, w2: np.ndarray) -> np.ndarray:
    """O4. SwiGLU expert FFN in float64: W2 (silu(W1 x) * (W3 x)).

    x [n][H]; w13 [2I][H] (W1 rows, then W3 rows); w2 [H][I]. No biases.
    """
    inter = w2.shape[1]
    a = x @ w13[:inter].T
    b = x @ w13[inter:].T
    return (silu(a) * b) @ w2.T


def moe_output(x: np.ndarray, idx: np.ndarray, gates: np.ndarray, expert_weights,
               tokens=None, experts=None) -> np.ndarray:
    """O5. y[t] = sum_j gate[t][j] * FFN_{idx[t][j]}(x[t]) in float64.

    x float64 [T][H]; expert_weights(e) -> (w13, w2) float64. `tokens`
    restricts the evaluation to a subset of token rows (returned in that order);
    `experts` restricts the sum to the routes of those experts (the partial sum
    a cost sample of the full output evaluates).
    """
    T = x.shape[0]
    rows = np.arange(T) if tokens is None else np.asarray(tokens)
    y = np.zeros((rows.size, x.shape[1]), dtype=np.float64)
    sub = idx[rows]
    todo = np.unique(sub)
    if experts is not None:
        todo = np.intersect1d(todo, np.asarray(experts))
    for e in todo:
        w13, w2 = expert_weights(int(e))
        for j in range(idx.shape[1]):
            sel = np.nonzero(sub[:, j] == e)[0]
            if sel.size:
                out = expert_ffn(x[rows[sel]], w13, w2)
                y[sel] += gates[rows[sel], j].astype(np.float64)[:, None] * out
    return y


# ---------------------------------------------------------------- O6 score
def score(idx: np.ndarray, gates: np.ndarray, conf: np.ndarray, n_experts: int):
    """O6/O7. Reuse-priority numerators of Sec. 4.3 with psi(c) = c.

    S[e] = sum over routes (t, j) with idx[t][j] == e of
           floor(float64(gate[t][j]) * float64(conf[t]) * 2^48).
    Experts routed by no token (stale residents included) get 0.
    Returns (S as Python ints in a uint64 array, p = S / sum(S) in float64).
    """
    conf = np.asarray(conf, dtype=np.float32)
    if not np.all((conf >= 0.0) & (conf <= 1.0)):
        raise ValueError("confidence outside [0, 1]")
    T, k = idx.shape
    S = [0] * n_experts
    for t in range(T):
        c = float(conf[t])
        for j in range(k):
            term = math.floor(float(gates[t, j]) * c * SCORE_SCALE)
            S[int(idx[t, j])] += int(term)
    total = sum(S)
    p = np.array([s / total if total else 0.0 for s in S], dtype=np.float64)
    return np.array(S, dtype=np.uint64), p


# --------------------------------------------------------------- O8 retain
def retain(S: np.ndarray, resident: np.ndarray, miss: np.ndarray, capacity: int):
    """O8. R^{i+1} = Top_C(R^i u G^i, p) with G = M (retention rule, Sec. 4.2).

    Candidates are ordered by (S desc, previously resident first, id asc) and
    the first min(C, |cand|) are kept. Returns the new resident mask (bool [E]).
    """
    resident = np.asarray(resident, dtype=bool)
    cand = [e for e in range(len(S)) if resident[e] or miss[e]]
    cand.sort(key=lambda e: (-int(S[e]), 0 if resident[e] else 1, e))
    keep = np.zeros(len(S), dtype=bool)
    for e in cand[: max(0, min(capacity, len(cand)))]:
        keep[e] = True
    return keep


# --------------------------------------------------- O1..O9, one layer-step
def layer_step(logits, conf, resident, top_k: int, capacity: int, policy: str = "priority",
               history=None):
    """Control path of one layer-iteration (O1-O3, O6-O8): no expert outputs.

    policy "priority" (the paper's) ranks the candidates by S; "lru" / "lfu"
    (O11) by the layer's history, which `history` (a PolicyHistory) carries
    from one iteration to the next. Returns a dict with idx, gates, counts,
    offsets, perm, inv_perm, active, hit, miss, n_hits, n_misses, util, S, p,
    the retention key and the new resident mask.
    """
    E = logits.shape[1]
    idx, gates = route(logits, top_k)
    counts, offsets, perm, inv_perm = permute(idx, E)
    active, hit, miss = classify(counts, resident)
    S, p = score(idx, gates, conf, E)
    if policy == "priority":
        key = S
    else:
        history.observe(counts)
        key = history.key(policy)
    new_res = retain(key, resident, miss, capacity)
    n_hits = int(hit.sum())
    return dict(idx=idx, gates=gates, counts=counts, offsets=offsets, perm=perm,
                inv_perm=inv_perm, active=active, hit=hit, miss=miss,
                n_active=int(active.sum()), n_hits=n_hits, n_misses=int(miss.sum()),
                util=(n_hits / capacity if capacity > 0 else 0.0),
                S=S, p=p, key=np.asarray(key, dtype=np.uint64),
                resident_before=np.asarray(resident, dtype=bool).copy(),
                resident_after=new_res)


def run_schedule(logits_fn, conf_fn, n_layers: int, n_iters: int, n_experts: int,
                 top_k: int, capacity: int, resident0=None, adapt_period: int = 0,
                 policy: str = "priority"):
    """O9. Replays the cache state of every layer over iterations 0..n_iters-1.

    logits_fn(l, i) -> float32 [T][E]; conf_fn(l, i) -> float32 [T].
    The cache starts empty (R^0 = {} per layer) unless resident0 is given.
    Every layer starts with capacity min(C, E). With adapt_period > 0 the
    capacities are re-sized (O10) after every adapt_period-th iteration.
    Returns steps[i][l] (the layer_step dicts, each with the `capacity` in
    effect). After an update, the last layer's dict of that iteration also
    holds `capacities_after` and `residents_after_update` (every layer's new
    capacity and resident mask). `policy` selects the retention key (O11).
    Each dict also holds `prev_transferred` (experts the layer transferred at
    its previous iteration) and `reused_transfers` (those of them retained and
    activated now), the terms of the effective transfer ratio.
    """
    if policy not in POLICIES:
        raise ValueError(f"unknown policy {policy}")
    res = [np.zeros(n_experts, dtype=bool) if resident0 is None
           else np.asarray(resident0[l], dtype=bool) for l in range(n_layers)]
    cap = [min(capacity, n_experts)] * n_layers
    stats = AdaptStats(n_layers)
    hist = [PolicyHistory(n_experts) for _ in range(n_layers)]
    prev_miss = [np.zeros(n_experts, dtype=bool) for _ in range(n_layers)]
    steps = []
    for i in range(n_iters):
        row = []
        for l in range(n_layers):
            st = layer_step(logits_fn(l, i), conf_fn(l, i), res[l], top_k, cap[l], policy, hist[l])
            st["capacity"] = cap[l]
            st["prev_transferred"] = int(prev_miss[l].sum())
            st["reused_transfers"] = int((st["active"] & st["resident_before"] & prev_miss[l]).sum())
            prev_miss[l] = st["miss"].copy()
            res[l] = st["resident_after"]
            if adapt_period > 0:
                stats.observe(l, st["n_active"], st["n_hits"], cap[l], n_experts)
            row.append(st)
        if adapt_period > 0 and (i + 1) % adapt_period == 0:
            cap = adapt_capacities(stats, n_layers * min(capacity, n_experts), n_experts, cap)
            res = [adapt_shrink(res[l], row[l]["key"], cap[l]) for l in range(n_layers)]
            row[-1]["capacities_after"] = list(cap)
            row[-1]["residents_after_update"] = [r.copy() for r in res]
        steps.append(row)
    return steps


# ------------------------------------------- O11 comparison retention policies
POLICIES = ("priority", "lru", "lfu")


class PolicyHistory:
    """History of one layer for LRU and LFU retention: the layer iteration in
    which each expert was last activated (iterations counted from 1; 0 never)
    and the routes sent to it so far."""

    def __init__(self, n_experts: int):
        self.iters = 0
        self.last_use = [0] * n_experts
        self.freq = [0] * n_experts

    def observe(self, counts):
        self.iters += 1
        for e, c in enumerate(counts):
            if c > 0:
                self.last_use[e] = self.iters
                self.freq[e] += int(c)

    def key(self, policy: str):
        return self.last_use if policy == "lru" else self.freq


def ideal_hits(n_active: int, capacity: int) -> int:
    """Clairvoyant ideal cache bound of one layer-iteration: knowing A, a cache
    of C experts holds min(C, |A|) of them when the layer runs."""
    return min(capacity, n_active)


def effective_transfer_ratio(steps) -> float:
    """Share of transferred experts retained and activated again at the next
    iteration of their layer (over transfers that have a next iteration)."""
    moved = sum(st["prev_transferred"] for row in steps for st in row)
    reused = sum(st["reused_transfers"] for row in steps for st in row)
    return reused / moved if moved else 0.0


# ------------------------------------------- O12 cooperative compensation
def coop_rho(t_h2d: float, tau_cpu: float, nbar: float) -> float:
    """Hardware-aware baseline share of misses to transfer (Sec. 4.4):
    rho = nbar tau_CPU / (nbar tau_CPU + T_H2D)."""
    cpu = nbar * tau_cpu
    den = cpu + t_h2d
    return cpu / den if den > 0.0 else 1.0


def coop_objective(G, misses, n_tok, S, S_total, t_h2d, tau_cpu, lam) -> float:
    """J(G) = T_comp(G) - lambda * sum_{e in G} p_e (Sec. 4.4), with
    T_comp = max(T_H2D |G|, tau_CPU * tokens left to the CPU)."""
    cpu_tokens = 0
    for e in misses:
        if e not in G:
            cpu_tokens += int(n_tok[e])
    t_comp = max(t_h2d * float(len(G)), tau_cpu * float(cpu_tokens))
    mass = 0
    for e in G:
        mass += int(S[e])
    share = float(mass) / float(S_total) if S_total > 0 else 0.0
    return t_comp - lam * share


def coop_dispatch(miss, n_tok, S, t_h2d: float, tau_cpu: float, nbar: float, lam: float):
    """O12. Which misses to transfer (Sec. 4.4). miss: bool [E]; n_tok: routed
    tokens per expert; S: priority numerators of every expert of the layer.
    Stage 1 takes the round_half_up(rho |M|) misses of highest priority;
    stage 2 makes bounded swaps that lower J. Returns the transfer mask G."""
    E = len(miss)
    misses = [e for e in range(E) if miss[e]]
    S_total = 0
    for e in range(E):
        S_total += int(S[e])
    rho = coop_rho(t_h2d, tau_cpu, nbar)
    n_g = int(math.floor(rho * float(len(misses)) + 0.5))
    by_priority = sorted(misses, key=lambda e: (-int(S[e]), e))
    G = set(by_priority[:n_g])
    J = coop_objective(G, misses, n_tok, S, S_total, t_h2d, tau_cpu, lam)
    for _ in range(len(misses)):
        best = None
        for g in sorted(G):
            for c in misses:
                if c in G:
                    continue
                Gs = (G - {g}) | {c}
                j = coop_objective(Gs, misses, n_tok, S, S_total, t_h2d, tau_cpu, lam)
                if best is None or j < best[0]:
                    best = (j, Gs)
        if best is None or not best[0] < J:
            break
        J, G = best
    out = np.zeros(E, dtype=bool)
    for e in G:
        out[e] = True
    return out


def coop_layer_step(logits, conf, resident, top_k: int, capacity: int, t_h2d: float,
                    tau_cpu: float, nbar: float, lam: float):
    """O1-O3, O6, O12, O8 for one layer-iteration with cooperative
    compensation: the misses are split into transfers G and CPU executions;
    the retention keeps Top_C of R u G. Returns the layer_step dict plus
    `transfer` (G) and `cpu` (M - G) masks."""
    E = logits.shape[1]
    idx, gates = route(logits, top_k)
    counts, offsets, perm, inv_perm = permute(idx, E)
    active, hit, miss = classify(counts, resident)
    S, p = score(idx, gates, conf, E)
    G = coop_dispatch(miss, counts, S, t_h2d, tau_cpu, nbar, lam)
    new_res = retain(S, resident, G, capacity)
    n_hits = int(hit.sum())
    return dict(idx=idx, gates=gates, counts=counts, offsets=offsets, perm=perm,
                inv_perm=inv_perm, active=active, hit=hit, miss=miss,
                n_active=int(active.sum()), n_hits=n_hits, n_misses=int(miss.sum()),
                util=(n_hits / capacity if capacity > 0 else 0.0), S=S, p=p,
                key=np.asarray(S, dtype=np.uint64),
                resident_before=np.asarray(resident, dtype=bool).copy(), resident_after=new_res,
                transfer=G, cpu=miss & ~G)


def run_coop_schedule(logits_fn, conf_fn, n_layers: int, n_iters: int, n_experts: int,
                      top_k: int, capacity: int, t_h2d: float, tau_cpu: float, nbar: float,
                      lam: float):
    """O9 with cooperative compensation (O12): steps[i][l]. Each dict also
    holds prev_transferred / reused_transfers over the transferred experts."""
    res = [np.zeros(n_experts, dtype=bool) for _ in range(n_layers)]
    prev = [np.zeros(n_experts, dtype=bool) for _ in range(n_layers)]
    cap = min(capacity, n_experts)
    steps = []
    for i in range(n_iters):
        row = []
        for l in range(n_layers):
            st = coop_layer_step(logits_fn(l, i), conf_fn(l, i), res[l], top_k, cap, t_h2d,
                                 tau_cpu, nbar, lam)
            st["capacity"] = cap
            st["prev_transferred"] = int(prev[l].sum())
            st["reused_transfers"] = int((st["active"] & st["resident_before"] & prev[l]).sum())
            prev[l] = st["transfer"].copy()
            res[l] = st["resident_after"]
            row.append(st)
        steps.append(row)
    return steps


# --------------------------------------------------------------- O13 gate
def router_logits(x: np.ndarray, w_gate: np.ndarray) -> np.ndarray:
    """O13. The gate's logits: logits[t][e] = sum_h x[t][h] * w_gate[e][h] in
    float64 (x [T][H], w_gate [E][H])."""
    return np.asarray(x, dtype=np.float64) @ np.asarray(w_gate, dtype=np.float64).T


def fp32_sum_bound(x: np.ndarray, w_gate: np.ndarray) -> np.ndarray:
    """Bound on |fl32 accumulation - exact| of each logit when the H products
    are exact and summed in float32 in any order: gamma_H * sum_h |x_h w_h|,
    gamma_n = n u / (1 - n u), u = 2^-24."""
    H = np.asarray(x).shape[1]
    u = 2.0 ** -24
    gamma = H * u / (1.0 - H * u)
    return gamma * (np.abs(np.asarray(x, np.float64)) @ np.abs(np.asarray(w_gate, np.float64)).T)


# ------------------------------------------------- O10 layer-adaptive sizing
class AdaptStats:
    """Smoothed per-layer statistics of Sec. 4.3: activation ratio a_l and
    expert-cache utilisation u_l, exponential moving averages with weight 1/2
    on the newest observation (float64)."""

    def __init__(self, n_layers: int):
        self.a = [0.0] * n_layers
        self.u = [0.0] * n_layers
        self.has_a = [False] * n_layers
        self.has_u = [False] * n_layers

    def observe(self, layer: int, n_active: int, n_hits: int, capacity: int, n_experts: int):
        a_obs = float(n_active) / float(n_experts)
        self.a[layer] = 0.5 * a_obs + 0.5 * self.a[layer] if self.has_a[layer] else a_obs
        self.has_a[layer] = True
        if capacity > 0:
            u_obs = float(n_hits) / float(capacity)
            self.u[layer] = 0.5 * u_obs + 0.5 * self.u[layer] if self.has_u[layer] else u_obs
            self.has_u[layer] = True

    def weights(self):
        """w_l = a_l * u_l (0 for a layer without a utilisation observation)."""
        return [self.a[l] * self.u[l] if (self.has_a[l] and self.has_u[l]) else 0.0
                for l in range(len(self.a))]


def adapt_capacities(stats: AdaptStats, c_total: int, n_experts: int, cap_old):
    """O10. C_l = C_total * w_l / sum_j w_j with w_l = a_l * u_l (Sec. 4.3), in
    integers: no layer above E (its share is re-spread over the others), then
    the largest remainder. Returns the new capacities (the old ones if every
    w_l is 0)."""
    w = stats.weights()
    L = len(w)
    total = 0.0
    for l in range(L):
        total += w[l]
    if total == 0.0:
        return list(cap_old)
    cap = [0] * L
    open_ = [True] * L
    avail = c_total
    q = [0.0] * L
    while True:
        W = 0.0
        for l in range(L):
            if open_[l]:
                W += w[l]
        if W == 0.0:
            for l in range(L):
                if open_[l]:
                    q[l] = 0.0
            break
        for l in range(L):
            if open_[l]:
                q[l] = (float(avail) * w[l]) / W
        over = [l for l in range(L) if open_[l] and q[l] > n_experts]
        if not over:
            break
        for l in over:
            cap[l] = n_experts
            open_[l] = False
            avail -= n_experts
    frac = [0.0] * L
    given = 0
    for l in range(L):
        if open_[l]:
            cap[l] = int(math.floor(q[l]))
            frac[l] = q[l] - math.floor(q[l])
            given += cap[l]
    left = avail - given
    order = sorted((l for l in range(L) if open_[l] and cap[l] < n_experts),
                   key=lambda l: (-frac[l], l))
    for l in order[:max(0, left)]:
        cap[l] += 1
    if left < 0:   # rounded shares summing above C_avail: take back from the smallest remainders
        back = sorted((l for l in range(L) if open_[l] and cap[l] > 0), key=lambda l: (frac[l], -l))
        for l in back[:-left]:
            cap[l] -= 1
    return cap


def adapt_shrink(resident: np.ndarray, S: np.ndarray, capacity: int) -> np.ndarray:
    """O10 enforcement: a layer over its new capacity keeps its `capacity`
    residents of highest priority, by (S desc, id asc), S the keys of its last
    retention (the priority numerators under the paper's policy); the rest are
    evicted."""
    resident = np.asarray(resident, dtype=bool)
    held = [e for e in range(len(resident)) if resident[e]]
    if len(held) <= capacity:
        return resident.copy()
    held.sort(key=lambda e: (-int(S[e]), e))
    keep = np.zeros(len(resident), dtype=bool)
    for e in held[:max(0, capacity)]:
        keep[e] = True
    return keep
