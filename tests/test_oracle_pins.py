"""Pins of the CPU oracle against facts that do not come from the oracle itself.

Each check_* function takes the oracle function(s) under test as arguments, so
the planted-mistake tests at the bottom can hand it a deliberately broken
variant and show that the pin catches it. Sources of truth used here:
brute force over subsets (routing, retention), Python's sorted() (stable
permutation), a 50-digit mpmath evaluation (gates, SiLU), exact rationals
(scores), scipy's softmax (gates as a renormalised full softmax), closed forms
(score mass, full residency, zero capacity) and a hand-derived worked example.
"""
import itertools
import json
import math
import os
from fractions import Fraction

import mpmath
import numpy as np
import pytest
from scipy.special import softmax

import oracle
from oracle import oled_oracle as O

HERE = os.path.dirname(os.path.abspath(__file__))
mpmath.mp.dps = 50


def _f32_nearest(v: mpmath.mpf) -> np.float32:
    """float32 nearest to a high-precision value (ties to even)."""
    f = np.float32(float(v))
    best, bestd = f, abs(mpmath.mpf(float(f)) - v)
    for cand in (np.nextafter(f, np.float32(-np.inf)), np.nextafter(f, np.float32(np.inf))):
        d = abs(mpmath.mpf(float(cand)) - v)
        if d < bestd or (d == bestd and (cand.view(np.uint32) & 1) == 0):
            best, bestd = cand, d
    return best


def _rand_logits(rng, T, E, discrete=False):
    if discrete:   # many ties
        return rng.integers(-2, 3, size=(T, E)).astype(np.float32)
    return rng.standard_normal((T, E)).astype(np.float32)


# ------------------------------------------------------------------ routing
def check_route_bruteforce(route, logits, k):
    """The top-k set is the max-sum k-subset, ties -> lexicographically smallest ids."""
    idx, gates = route(logits, k)
    T, E = logits.shape
    for t in range(T):
        vals = [Fraction(float(v)) for v in logits[t]]
        best = None
        for sub in itertools.combinations(range(E), k):
            key = (sum(vals[e] for e in sub), tuple(-e for e in sub))
            if best is None or key > best[0]:
                best = (key, sub)
        assert sorted(int(e) for e in idx[t]) == list(best[1]), (t, idx[t], best[1])
        # slot order: logit non-increasing, equal logits by ascending id
        for j in range(k - 1):
            a, b = int(idx[t, j]), int(idx[t, j + 1])
            assert vals[a] > vals[b] or (vals[a] == vals[b] and a < b)


def check_gates_invariants(route, logits, k):
    idx, gates = route(logits, k)
    assert gates.dtype == np.float32
    assert np.all(gates > 0)
    assert np.all(np.diff(gates.astype(np.float64), axis=1) <= 0)
    s = gates.astype(np.float64).sum(axis=1)
    assert np.all(np.abs(s - 1.0) <= k * 2.0 ** -24), s


def check_gates_mpmath(route, logits, k):
    """Each gate is the float32 nearest to exp(l_j - l_0) / sum exp, at 50 digits."""
    idx, gates = route(logits, k)
    for t in range(logits.shape[0]):
        sel = [mpmath.mpf(float(logits[t, e])) for e in idx[t]]
        ex = [mpmath.exp(v - sel[0]) for v in sel]
        tot = mpmath.fsum(ex)
        for j in range(k):
            assert gates[t, j] == _f32_nearest(ex[j] / tot), (t, j)


def check_gates_full_softmax(route, logits, k):
    """Renormalised top-k of a full softmax (scipy) equals the gates within 1 ulp."""
    idx, gates = route(logits, k)
    full = softmax(logits.astype(np.float64), axis=1)
    sel = np.take_along_axis(full, idx.astype(np.int64), axis=1)
    ref = (sel / sel.sum(axis=1, keepdims=True)).astype(np.float32)
    ulp = np.abs(gates.view(np.int32).astype(np.int64) - ref.view(np.int32).astype(np.int64))
    assert ulp.max() <= 1, ulp.max()


@pytest.mark.parametrize("seed", range(6))
def test_route_bruteforce(seed):
    rng = np.random.default_rng(seed)
    E = int(rng.integers(2, 9))
    k = int(rng.integers(1, min(E, 4) + 1))
    T = int(rng.integers(1, 17))
    check_route_bruteforce(O.route, _rand_logits(rng, T, E, discrete=seed % 2 == 0), k)


def test_route_bruteforce_tiny_workload():
    from paper_2609_33385_amd import workload as W
    w = W.WORKLOADS[1]
    for it in range(w.n_iters):
        check_route_bruteforce(O.route, W.logits(w, 0, 0, 0, it), w.top_k)


@pytest.mark.parametrize("seed", range(4))
def test_gates(seed):
    rng = np.random.default_rng(100 + seed)
    T, E, k = 12, 16, [1, 2, 4, 8][seed]
    lg = (3.0 * rng.standard_normal((T, E))).astype(np.float32)
    check_gates_invariants(O.route, lg, k)
    check_gates_mpmath(O.route, lg, k)
    check_gates_full_softmax(O.route, lg, k)


def test_gates_special_cases():
    rng = np.random.default_rng(7)
    lg = rng.standard_normal((5, 8)).astype(np.float32)
    _, g = O.route(lg, 1)
    assert np.all(g == 1.0)                       # k = 1: the gate is exactly 1
    for k in (2, 4, 8):                           # equal logits: exactly 1/k
        _, g = O.route(np.full((3, 8), 0.7, np.float32), k)
        assert np.all(g == np.float32(1.0 / k))
    # -0.0 and +0.0 are equal logits: the tie goes to the lower id
    idx, _ = O.route(np.array([[-0.0, 0.0, -1.0]], np.float32), 1)
    assert idx[0, 0] == 0
    idx, _ = O.route(np.array([[-1.0, 0.0, -0.0]], np.float32), 1)
    assert idx[0, 0] == 1
    with pytest.raises(ValueError):
        O.route(np.array([[np.nan, 0.0]], np.float32), 1)


# -------------------------------------------------------------- permutation
def check_permute_sorted(permute, idx, E):
    counts, offsets, perm, inv_perm = permute(idx, E)
    flat = [int(e) for e in np.asarray(idx).ravel()]
    ref = sorted(range(len(flat)), key=lambda r: (flat[r], r))
    assert list(perm) == ref
    assert [int(c) for c in counts] == [flat.count(e) for e in range(E)]
    assert list(offsets) == [0] + list(itertools.accumulate(flat.count(e) for e in range(E)))
    assert all(perm[inv_perm[r]] == r for r in range(len(flat)))


@pytest.mark.parametrize("seed", range(6))
def test_permute(seed):
    rng = np.random.default_rng(200 + seed)
    E = int(rng.integers(1, 40))
    k = int(rng.integers(1, min(E, 8) + 1))
    T = int(rng.integers(1, 70))
    idx, _ = O.route(_rand_logits(rng, T, E, discrete=seed % 2 == 1), k)
    check_permute_sorted(O.permute, idx, E)


# ------------------------------------------------------------------- scores
def check_score_exact(score, idx, gates, conf, E):
    """S[e] equals the exact rational floor(g*c*2^48) summed per expert."""
    S, p = score(idx, gates, conf, E)
    ref = [0] * E
    for t in range(idx.shape[0]):
        for j in range(idx.shape[1]):
            ref[int(idx[t, j])] += math.floor(Fraction(float(gates[t, j])) *
                                              Fraction(float(conf[t])) * 2 ** 48)
    assert [int(s) for s in S] == ref


def check_score_mass(score, idx, gates, conf, E):
    """Closed form of the normaliser: sum_e S_e / 2^48 = sum_t c_t (gates sum to 1)."""
    S, p = score(idx, gates, conf, E)
    T, k = idx.shape
    tot = sum(int(s) for s in S) / 2.0 ** 48
    csum = float(np.sum(conf.astype(np.float64)))
    assert abs(tot - csum) <= csum * k * 2.0 ** -24 + T * k * 2.0 ** -48 + 1e-15
    if tot > 0:
        assert abs(p.sum() - 1.0) < 1e-12


@pytest.mark.parametrize("seed", range(4))
def test_score(seed):
    rng = np.random.default_rng(300 + seed)
    T, E, k = 40, 12, 3
    idx, gates = O.route(_rand_logits(rng, T, E), k)
    conf = rng.uniform(0, 1, T).astype(np.float32)
    check_score_exact(O.score, idx, gates, conf, E)
    check_score_mass(O.score, idx, gates, conf, E)
    # shuffling tokens leaves S unchanged
    sh = rng.permutation(T)
    S0, _ = O.score(idx, gates, conf, E)
    S1, _ = O.score(idx[sh], gates[sh], conf[sh], E)
    assert np.array_equal(S0, S1)


def test_score_special_cases():
    rng = np.random.default_rng(9)
    lg = rng.standard_normal((1, 6)).astype(np.float32)
    idx, g = O.route(lg, 3)
    _, p = O.score(idx, g, np.array([0.7], np.float32), 6)
    for j in range(3):                     # one token: p_e is its gate
        assert abs(p[idx[0, j]] - float(g[0, j])) < 1e-12
    assert all(p[e] == 0 for e in range(6) if e not in idx[0])
    # confidence identically 0: every priority is 0
    S, p = O.score(idx, g, np.array([0.0], np.float32), 6)
    assert int(S.sum()) == 0 and np.all(p == 0)
    with pytest.raises(ValueError):
        O.score(idx, g, np.array([1.5], np.float32), 6)


# ---------------------------------------------------------------- retention
def check_retain_bruteforce(retain, S, resident, miss, C):
    """Top-C: the unique subset whose every member outranks every non-member."""
    E = len(S)
    keep = retain(S, resident, miss, C)
    cand = [e for e in range(E) if resident[e] or miss[e]]
    key = {e: (int(S[e]), 1 if resident[e] else 0, -e) for e in cand}
    n = min(max(C, 0), len(cand))
    winners = [set(sub) for sub in itertools.combinations(cand, n)
               if all(key[a] > key[b] for a in sub for b in cand if b not in sub)]
    assert len(winners) == 1
    assert set(np.nonzero(keep)[0].tolist()) == winners[0]


@pytest.mark.parametrize("seed", range(8))
def test_retain_bruteforce(seed):
    rng = np.random.default_rng(400 + seed)
    E = int(rng.integers(1, 9))
    resident = rng.random(E) < 0.4
    miss = (rng.random(E) < 0.5) & ~resident
    # small score alphabet: many ties, including zero scores of stale residents
    S = rng.integers(0, 3, E).astype(np.uint64)
    S[~(miss | (rng.random(E) < 0.5))] = 0
    for C in range(0, E + 2):
        check_retain_bruteforce(O.retain, S, resident, miss, C)


# ------------------------------------------------------- schedule invariants
def _schedule(seed, T=12, E=8, k=2, C=3, L=2, N=6):
    rng = np.random.default_rng(seed)
    base = rng.standard_normal((L, T, E)) * 2
    steps = rng.standard_normal((N, L, T, E)) * 0.6
    lg = np.cumsum(steps, axis=0) + base[None]
    conf = rng.uniform(0, 1, (N, T)).astype(np.float32)
    return O.run_schedule(lambda l, i: lg[i, l].astype(np.float32), lambda l, i: conf[i],
                          L, N, E, k, C)


@pytest.mark.parametrize("C", [0, 1, 3, 5, 8, 10])
def test_schedule_invariants(C):
    E = 8
    steps = _schedule(500 + C, E=E, C=C)
    for row in steps:
        for st in row:
            R0, R1, A = st["resident_before"], st["resident_after"], st["active"]
            assert st["n_hits"] + st["n_misses"] == st["n_active"]
            assert st["n_hits"] <= R0.sum() <= max(C, 0) or C >= E
            assert R1.sum() == min(C, (R0 | A).sum())
            assert not np.any(R1 & ~(R0 | A))          # R' subset of R u A
            key = lambda e: (int(st["S"][e]), int(R0[e]), -e)
            kept = [e for e in range(E) if R1[e]]
            dropped = [e for e in range(E) if (R0[e] or A[e]) and not R1[e]]
            assert all(key(a) > key(b) for a in kept for b in dropped)
            assert np.all(st["S"][~A] == 0)              # stale residents score 0


def test_schedule_full_residency_closed_form():
    """C = E: the cache only grows; misses are first activations, hits re-activations."""
    E, L = 8, 2
    steps = _schedule(600, E=E, C=E, L=L)
    for l in range(L):
        seen = np.zeros(E, dtype=bool)
        for row in steps:
            st = row[l]
            assert st["n_hits"] == int((st["active"] & seen).sum())
            assert st["n_misses"] == int((st["active"] & ~seen).sum())
            seen |= st["active"]
            assert np.array_equal(st["resident_after"], seen)


def test_schedule_zero_capacity():
    steps = _schedule(700, C=0)
    for row in steps:
        for st in row:
            assert st["n_hits"] == 0 and st["n_misses"] == st["n_active"]
            assert not st["resident_after"].any()


# ------------------------------------------------------------ worked example
def test_worked_example():
    with open(os.path.join(HERE, "golden", "worked_example.json")) as f:
        ex = json.load(f)
    E, k, C = ex["n_experts"], ex["top_k"], ex["capacity"]
    lg = np.array(ex["logits"], np.float32)
    conf = np.array(ex["conf"], np.float32)
    res = np.zeros(E, bool)
    res[ex["resident_before"]] = True
    st = O.layer_step(lg, conf, res, k, C)
    want = ex["expect"]
    assert st["idx"].tolist() == want["idx"]
    assert st["counts"].tolist() == want["counts"]
    assert st["offsets"].tolist() == want["offsets"]
    assert st["perm"].tolist() == want["perm"]
    assert st["inv_perm"].tolist() == want["inv_perm"]
    assert np.nonzero(st["active"])[0].tolist() == want["active"]
    assert np.nonzero(st["hit"])[0].tolist() == want["hits"]
    assert np.nonzero(st["miss"])[0].tolist() == want["misses"]
    assert np.nonzero(st["resident_after"])[0].tolist() == want["resident_after"]
    order = sorted(range(E), key=lambda e: -int(st["S"][e]))
    assert order == want["score_rank"]
    assert st["n_hits"] == 1 and st["n_misses"] == 3 and abs(st["util"] - 1 / 3) < 1e-15
    # gates at 50 digits: 1/(1+e^-1), 1/2, 1/(1+e^-1.5) and complements
    g_ref = [[1 / (1 + mpmath.e ** -1), mpmath.e ** -1 / (1 + mpmath.e ** -1)],
             [mpmath.mpf(1) / 2, mpmath.mpf(1) / 2],
             [1 / (1 + mpmath.e ** -1.5), mpmath.e ** -1.5 / (1 + mpmath.e ** -1.5)]]
    g32 = np.array([[_f32_nearest(v) for v in row] for row in g_ref], np.float32)
    assert np.array_equal(st["gates"], g32)
    # scores from the reference gates in exact rationals
    S_ref = [0] * E
    for t in range(3):
        for j in range(k):
            S_ref[want["idx"][t][j]] += math.floor(Fraction(float(g32[t, j])) *
                                                   Fraction(float(conf[t])) * 2 ** 48)
    assert [int(s) for s in st["S"]] == S_ref
    assert S_ref[4] == 0


# ------------------------------------------------------------- expert FFN
def check_ffn_hand(expert_ffn):
    """H = I = 2 with distinct, non-symmetric matrices, evaluated by hand.

    W1 = [[1,0],[0,2]], W3 = [[0,1],[1,0]], W2 = [[1,2],[3,4]], x = [1,-1]:
    W1 x = [1,-2], W3 x = [-1,1], h = [-silu(1), silu(-2)],
    y = [h0 + 2 h1, 3 h0 + 4 h1].
    """
    w13 = np.array([[1, 0], [0, 2], [0, 1], [1, 0]], np.float64)
    w2 = np.array([[1, 2], [3, 4]], np.float64)
    y = expert_ffn(np.array([[1.0, -1.0]]), w13, w2)[0]
    s1 = 1 / (1 + mpmath.e ** -1)          # silu(1) = 1 * sigmoid(1)
    sm2 = -2 / (1 + mpmath.e ** 2)         # silu(-2)
    h0, h1 = -s1, sm2 * 1
    ref = [h0 + 2 * h1, 3 * h0 + 4 * h1]
    assert abs(y[0] - float(ref[0])) < 1e-14 and abs(y[1] - float(ref[1])) < 1e-14, (y, ref)


def test_ffn_hand():
    check_ffn_hand(O.expert_ffn)


def check_moe_dense(moe_output, route):
    """k = E: the layer is the softmax-weighted sum of every expert (scipy softmax)."""
    rng = np.random.default_rng(11)
    T, E, H, I = 5, 4, 6, 3
    lg = rng.standard_normal((T, E)).astype(np.float32)
    x = rng.standard_normal((T, H))
    Ws = [(rng.standard_normal((2 * I, H)), rng.standard_normal((H, I))) for _ in range(E)]
    idx, g = route(lg, E)
    y = moe_output(x, idx, g, lambda e: Ws[e])
    sm = softmax(lg.astype(np.float64), axis=1)
    for t in range(T):
        ref = np.zeros(H)
        for e in range(E):
            w13, w2 = Ws[e]
            a = np.array([sum(w13[i, c] * x[t, c] for c in range(H)) for i in range(I)])
            b = np.array([sum(w13[I + i, c] * x[t, c] for c in range(H)) for i in range(I)])
            h = a / (1 + np.exp(-a)) * b
            ref += sm[t, e] * np.array([sum(w2[r, i] * h[i] for i in range(I)) for r in range(H)])
        assert np.allclose(y[t], ref, rtol=1e-6, atol=1e-9)


def test_moe_dense():
    check_moe_dense(O.moe_output, O.route)


def test_moe_token_subset():
    rng = np.random.default_rng(12)
    T, E, H, I, k = 9, 5, 4, 3, 2
    lg = rng.standard_normal((T, E)).astype(np.float32)
    x = rng.standard_normal((T, H))
    Ws = [(rng.standard_normal((2 * I, H)), rng.standard_normal((H, I))) for _ in range(E)]
    idx, g = O.route(lg, k)
    y = O.moe_output(x, idx, g, lambda e: Ws[e])
    sub = [7, 0, 3]
    ys = O.moe_output(x, idx, g, lambda e: Ws[e], tokens=sub)
    assert np.allclose(ys, y[sub], rtol=1e-13, atol=1e-15)


def test_moe_expert_subsets_partition_the_output():
    """Partial sums over disjoint expert sets add up to the full output, and
    one expert's partial sum is its gate-weighted FFN on its own tokens."""
    rng = np.random.default_rng(13)
    T, E, H, I, k = 11, 6, 4, 3, 3
    lg = rng.standard_normal((T, E)).astype(np.float32)
    x = rng.standard_normal((T, H))
    Ws = [(rng.standard_normal((2 * I, H)), rng.standard_normal((H, I))) for _ in range(E)]
    idx, g = O.route(lg, k)
    y = O.moe_output(x, idx, g, lambda e: Ws[e])
    parts = [O.moe_output(x, idx, g, lambda e: Ws[e], experts=s) for s in ([0, 3], [1, 5], [2, 4])]
    assert np.allclose(sum(parts), y, rtol=1e-12, atol=1e-14)
    e = int(idx[0, 0])
    ye = O.moe_output(x, idx, g, lambda q: Ws[q], experts=[e])
    for t in range(T):
        want = np.zeros(H)
        for j in range(k):
            if idx[t, j] == e:
                want += float(g[t, j]) * O.expert_ffn(x[t:t + 1], *Ws[e])[0]
        assert np.allclose(ye[t], want, rtol=1e-12, atol=1e-14)


def test_bf16_decode():
    bits = np.array([0x3F80, 0xBF80, 0x0000, 0x8000, 0x4049, 0x7F7F], np.uint16)
    v = oracle.bf16_bits_to_f64(bits)
    assert v[0] == 1.0 and v[1] == -1.0 and v[2] == 0.0
    assert v[4] == 3.140625
    assert v[5] == float(Fraction(2) ** 127 * (2 - Fraction(1, 2 ** 7)))


# ----------------------------------------------- planted mistakes get caught
def _bad_route_tie_high(logits, k):
    T, E = logits.shape
    idx = np.argsort(-logits.astype(np.float64)[:, ::-1], axis=1, kind="stable")
    idx = (E - 1 - idx[:, :k]).astype(np.int32)
    return idx, O.route(logits, k)[1]


def _bad_route_drop_term(logits, k):
    idx, _ = O.route(logits, k)
    g = np.empty(idx.shape, np.float32)
    for t in range(idx.shape[0]):
        sel = [float(logits[t, e]) for e in idx[t]]
        ex = [math.exp(v - sel[0]) for v in sel]
        s = sum(ex[:-1]) if k > 1 else ex[0]
        g[t] = [np.float32(v / s) for v in ex]
    return idx, g


def _bad_permute_jmajor(idx, E):
    T, k = idx.shape
    return O.permute(np.ascontiguousarray(idx.T), E)[:1] + tuple(
        _remap(O.permute(np.ascontiguousarray(idx.T), E), T, k)[1:])


def _remap(res, T, k):
    counts, offsets, perm, inv = res
    # position order built from j-major routes, relabelled as t*k+j
    relabel = np.array([(r % T) * k + r // T for r in range(T * k)])
    return counts, offsets, relabel[perm], None


def _bad_score_no_conf(idx, gates, conf, E):
    return O.score(idx, gates, np.ones_like(conf), E)


def _bad_retain_extra(S, resident, miss, C):
    return O.retain(S, resident, miss, C + 1)


def _bad_retain_no_resident_tiebreak(S, resident, miss, C):
    return O.retain(S, np.zeros_like(resident), miss | resident, C)


def _bad_ffn_swap13(x, w13, w2):
    I = w2.shape[1]
    return O.expert_ffn(x, np.concatenate([w13[I:], w13[:I]]), w2)


def _bad_ffn_transpose_w2(x, w13, w2):
    return O.expert_ffn(x, w13, np.ascontiguousarray(w2.T))


def test_planted_mistakes_are_caught():
    rng = np.random.default_rng(13)
    lg = _rand_logits(rng, 10, 6, discrete=True)
    with pytest.raises(AssertionError):
        check_route_bruteforce(_bad_route_tie_high, lg, 2)
    lg2 = (2 * rng.standard_normal((6, 8))).astype(np.float32)
    with pytest.raises(AssertionError):
        check_gates_invariants(_bad_route_drop_term, lg2, 4)
    idx, g = O.route(_rand_logits(rng, 12, 5), 2)
    with pytest.raises(AssertionError):
        counts, offsets, perm, _ = _bad_permute_jmajor(idx, 5)
        check_permute_sorted(lambda i, E: (counts, offsets, perm, np.argsort(perm)), idx, 5)
    conf = rng.uniform(0, 0.9, 12).astype(np.float32)
    with pytest.raises(AssertionError):
        check_score_mass(_bad_score_no_conf, idx, g, conf, 5)
    S = np.array([3, 1, 0, 2, 0, 0], np.uint64)
    res = np.array([0, 1, 1, 0, 0, 1], bool)
    miss = np.array([1, 0, 0, 1, 0, 0], bool)
    with pytest.raises(AssertionError):
        check_retain_bruteforce(_bad_retain_extra, S, res, miss, 3)
    # zero-score tie between a miss (id 1, confidence 0) and a resident (id 4)
    S0 = np.array([3, 0, 0, 2, 0, 0], np.uint64)
    res0 = np.array([0, 0, 0, 0, 1, 0], bool)
    miss0 = np.array([1, 1, 0, 1, 0, 0], bool)
    check_retain_bruteforce(O.retain, S0, res0, miss0, 3)
    with pytest.raises(AssertionError):
        check_retain_bruteforce(_bad_retain_no_resident_tiebreak, S0, res0, miss0, 3)
    with pytest.raises(AssertionError):
        check_ffn_hand(_bad_ffn_swap13)
    with pytest.raises(AssertionError):
        check_ffn_hand(_bad_ffn_transpose_w2)
