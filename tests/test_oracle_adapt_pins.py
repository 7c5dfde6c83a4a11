"""Pins of the oracle's layer-adaptive cache sizing (O10) against facts that do
not come from the oracle: the closed form of an exponential moving average with
weight 1/2, brute force over integer capacity vectors (the largest-remainder
allocation is the integer vector with the given sum closest to the shares),
hand-worked water-filling cases, brute force over subsets for the eviction,
and invariants of whole schedules. As in the other pin file, every check_*
takes the function under test, and planted mistakes are shown to fail.
"""
import itertools
from fractions import Fraction

import numpy as np
import pytest

from oracle import oled_oracle as O


# ------------------------------------------------------------- smoothing
def ema_closed_form(obs):
    """x_0 = o_0, x_n = o_n/2 + x_{n-1}/2, written out: the newest observation
    weighs 1/2, the one before 1/4, ..., and the first one 1/2^n."""
    n = len(obs) - 1
    x = Fraction(obs[0]) / (2 ** n)
    for j in range(1, n + 1):
        x += Fraction(obs[j]) / (2 ** (n - j + 1))
    return x


def check_ema(stats_cls, seq, E, C):
    """seq: [(n_active, n_hits, capacity)] of one layer."""
    st = stats_cls(1)
    a_obs, u_obs = [], []
    for n_act, n_hit, cap in seq:
        st.observe(0, n_act, n_hit, cap, E)
        a_obs.append(Fraction(n_act, E))
        if cap > 0:
            u_obs.append(Fraction(n_hit, cap))
        assert Fraction(st.a[0]) == ema_closed_form(a_obs)
        if u_obs:
            assert Fraction(st.u[0]) == ema_closed_form(u_obs)
        else:
            assert not st.has_u[0]


def test_ema_closed_form():
    # dyadic observations (E and capacities powers of two): float64 is exact
    check_ema(O.AdaptStats, [(8, 2, 4), (0, 4, 4), (4, 0, 4), (6, 1, 4), (7, 3, 4)], 8, 4)
    check_ema(O.AdaptStats, [(3, 0, 0), (5, 2, 2), (1, 1, 2)], 8, 2)   # capacity 0 skips u


def test_ema_hand_values():
    st = O.AdaptStats(2)
    for n_act, n_hit in ((8, 2), (0, 4), (4, 0)):
        st.observe(1, n_act, n_hit, 4, 8)
    assert (st.a[1], st.u[1]) == (0.5, 0.375)   # a: 1, 0.5, 0.5; u: 0.5, 0.75, 0.375
    assert not st.has_a[0] and st.weights()[0] == 0.0
    assert st.weights()[1] == 0.5 * 0.375


# ------------------------------------------------- capacities from weights
def _stats(a, u):
    st = O.AdaptStats(len(a))
    st.a, st.u = list(a), list(u)
    st.has_a = [True] * len(a)
    st.has_u = [True] * len(a)
    return st


def exact_shares(w, c_total, E):
    """Water-filling in exact rationals: shares proportional to w, none above E."""
    L = len(w)
    q = [Fraction(0)] * L
    open_ = [True] * L
    avail = Fraction(c_total)
    while True:
        W = sum(Fraction(w[l]) for l in range(L) if open_[l])
        if W == 0:
            break
        sh = {l: avail * Fraction(w[l]) / W for l in range(L) if open_[l]}
        over = [l for l in sh if sh[l] > E]
        if not over:
            for l, v in sh.items():
                q[l] = v
            break
        for l in over:
            q[l] = Fraction(E)
            open_[l] = False
            avail -= E
    return q


def brute_capacities(w, c_total, E):
    """The integer vector c (0 <= c_l <= E, sum c = sum of the exact shares)
    closest to the exact shares in squared distance; among equally close ones
    the lexicographically largest (the lower layer gets the unit)."""
    q = exact_shares(w, c_total, E)
    target = sum(q)
    assert target.denominator == 1
    best = None
    for c in itertools.product(range(E + 1), repeat=len(w)):
        if sum(c) != target:
            continue
        d = sum((Fraction(ci) - qi) ** 2 for ci, qi in zip(c, q))
        key = (-d, c)
        if best is None or key > best[0]:
            best = (key, list(c))
    return best[1]


def _well_separated(w, c_total, E):
    """Exact fractional parts far from each other and from 0 and 1, so that the
    float64 shares order them as the exact ones do."""
    q = exact_shares(w, c_total, E)
    fr = [float(x - (x.numerator // x.denominator)) for x in q if x < E]
    for f in fr:
        if f < 1e-9 or f > 1 - 1e-9:
            return False
    return all(abs(a - b) > 1e-9 for a, b in itertools.combinations(fr, 2))


def check_capacities_bruteforce(adapt_capacities, a, u, c_total, E):
    st = _stats(a, u)
    got = adapt_capacities(st, c_total, E, [0] * len(a))
    want = brute_capacities([Fraction(x) * Fraction(y) for x, y in zip(a, u)], c_total, E)
    assert got == want, (a, u, c_total, E, got, want)


@pytest.mark.parametrize("seed", range(40))
def test_capacities_bruteforce(seed):
    rng = np.random.default_rng(seed)
    L = int(rng.integers(2, 5))
    E = int(rng.integers(2, 6))
    c_total = int(rng.integers(1, L * E + 1))
    for _ in range(50):
        a = [float(v) for v in rng.integers(1, 9, L) / 8.0]
        u = [float(v) for v in rng.integers(0, 9, L) / 8.0]
        if sum(u) == 0 or not _well_separated([x * y for x, y in zip(a, u)], c_total, E):
            continue
        check_capacities_bruteforce(O.adapt_capacities, a, u, c_total, E)
        return
    pytest.skip("no well-separated draw")


def test_capacities_ties_go_to_lower_layers():
    # four equal weights, 6 units: shares 1.5 each, the two lower layers round up
    assert O.adapt_capacities(_stats([0.5] * 4, [0.5] * 4), 6, 8, [0] * 4) == [2, 2, 1, 1]
    # equal fractional parts across different shares (0.5 and 1.5)
    assert O.adapt_capacities(_stats([0.25, 0.75], [1.0, 1.0]), 2, 8, [0, 0]) == [1, 1]


def test_capacities_water_filling():
    # shares 4.8, 0.6, 0.6 of 6 with E = 4: layer 0 is capped, 2 units re-shared
    assert O.adapt_capacities(_stats([1.0, 0.125, 0.125], [1.0, 1.0, 1.0]), 6, 4, [0] * 3) == [4, 1, 1]
    # two rounds: 10 units over weights 8, 4, 1, 1 with E = 4
    #   first: 5.71, 2.86, 0.71, 0.71 -> layer 0 capped; then 6 over 4, 1, 1: 4, 1, 1
    assert O.adapt_capacities(_stats([1.0, 0.5, 0.125, 0.125], [1.0] * 4), 10, 4, [0] * 4) == [4, 4, 1, 1]
    # room for everything: every layer at E
    assert O.adapt_capacities(_stats([1.0, 0.5], [1.0, 1.0]), 8, 4, [0, 0]) == [4, 4]


def test_capacities_special_cases():
    # homogeneous layers keep the uniform split
    assert O.adapt_capacities(_stats([0.3] * 5, [0.7] * 5), 5 * 26, 64, [26] * 5) == [26] * 5
    # no information (all weights zero): unchanged
    assert O.adapt_capacities(_stats([0.5, 0.5], [0.0, 0.0]), 8, 8, [3, 5]) == [3, 5]
    # a layer with zero weight gets nothing while the others have room
    assert O.adapt_capacities(_stats([0.5, 0.5, 0.5], [1.0, 0.0, 0.5]), 6, 8, [2, 2, 2]) == [4, 0, 2]
    # one layer: all of C_total, at most E
    assert O.adapt_capacities(_stats([0.2], [0.9]), 7, 8, [7]) == [7]


@pytest.mark.parametrize("seed", range(10))
def test_capacities_invariants(seed):
    rng = np.random.default_rng(100 + seed)
    L, E = int(rng.integers(2, 40)), int(rng.integers(4, 129))
    c_total = int(rng.integers(0, L * E + 1))
    a = list(rng.uniform(0, 1, L))
    u = list(rng.uniform(0, 1, L) * (rng.uniform(0, 1, L) > 0.2))
    cap = O.adapt_capacities(_stats(a, u), c_total, E, [0] * L)
    w = [x * y for x, y in zip(a, u)]
    assert all(0 <= c <= E for c in cap)
    assert sum(cap) <= c_total
    if sum(w) > 0 and c_total <= E * sum(1 for x in w if x > 0):
        assert sum(cap) == c_total
    for i in range(L):
        if w[i] == 0 and sum(w) > 0 and c_total <= E * sum(1 for x in w if x > 0):
            assert cap[i] == 0
        for j in range(L):
            if w[i] > w[j] * (1 + 1e-9):
                assert cap[i] >= cap[j]


# -------------------------------------------------------------- eviction
def check_shrink_bruteforce(shrink, S, resident, cap):
    got = shrink(resident, S, cap)
    held = [e for e in range(len(S)) if resident[e]]
    if len(held) <= cap:
        assert np.array_equal(got, resident)
        return
    best = None
    for sub in itertools.combinations(held, cap):
        key = sorted(((int(S[e]), -e) for e in sub), reverse=True)
        if best is None or key > best[0]:
            best = (key, set(sub))
    assert {e for e in range(len(S)) if got[e]} == best[1]


@pytest.mark.parametrize("seed", range(10))
def test_shrink_bruteforce(seed):
    rng = np.random.default_rng(200 + seed)
    E = int(rng.integers(3, 9))
    S = rng.integers(0, 4, E).astype(np.uint64)     # small alphabet: many ties
    res = rng.uniform(0, 1, E) < 0.7
    for cap in range(0, E + 1):
        check_shrink_bruteforce(O.adapt_shrink, S, res, cap)


# ------------------------------------------------------ whole schedules
def _hetero_schedule(seed, period, T=16, E=8, k=2, C=3, L=4, N=12):
    """Layers with different routing spread: layer l's tokens share a preference
    of strength 0.5 + l, so low layers activate many experts and high ones few."""
    rng = np.random.default_rng(seed)
    z = rng.standard_normal((L, E))
    base = np.stack([(0.5 + l) * z[l][None, :] + rng.standard_normal((T, E)) for l in range(L)])
    steps = rng.standard_normal((N, L, T, E)) * 0.4
    lg = np.cumsum(steps, axis=0) + base[None]
    conf = rng.uniform(0, 1, (N, T)).astype(np.float32)
    run = lambda p: O.run_schedule(lambda l, i: lg[i, l].astype(np.float32), lambda l, i: conf[i],
                                   L, N, E, k, C, adapt_period=p)
    return run(period), run(0)


@pytest.mark.parametrize("period", [1, 2, 5])
def test_adaptive_schedule_invariants(period):
    E, C, L = 8, 3, 4
    steps, _ = _hetero_schedule(900 + period, period, E=E, C=C, L=L)
    cap = [C] * L
    changed = False
    for i, row in enumerate(steps):
        for l, st in enumerate(row):
            assert st["capacity"] == cap[l]
            R0, R1, A = st["resident_before"], st["resident_after"], st["active"]
            assert R0.sum() <= cap[l] and R1.sum() <= cap[l]
            assert R1.sum() == min(cap[l], (R0 | A).sum())
            assert not np.any(R1 & ~(R0 | A))
        last = row[-1]
        if (i + 1) % period == 0:
            new = last["capacities_after"]
            assert sum(new) <= C * L and all(0 <= c <= E for c in new)
            res = last["residents_after_update"]
            assert sum(int(r.sum()) for r in res) <= C * L
            for l in range(L):
                assert res[l].sum() == min(row[l]["resident_after"].sum(), new[l])
                assert not np.any(res[l] & ~row[l]["resident_after"])
            changed |= new != cap
            cap = new
        else:
            assert "capacities_after" not in last
    assert changed   # the layers differ, so capacity moves


def test_adaptive_schedule_special_cases():
    # a period beyond the schedule never updates: the fixed schedule
    steps, fixed = _hetero_schedule(950, 50)
    for r0, r1 in zip(steps, fixed):
        for a, b in zip(r0, r1):
            assert np.array_equal(a["resident_after"], b["resident_after"])
    # one layer holds all of C_total at every update: the fixed schedule
    rng = np.random.default_rng(3)
    lg = np.cumsum(rng.standard_normal((9, 1, 10, 6)), axis=0).astype(np.float32)
    conf = rng.uniform(0, 1, (9, 10)).astype(np.float32)
    run = lambda p: O.run_schedule(lambda l, i: lg[i, l], lambda l, i: conf[i], 1, 9, 6, 2, 3,
                                   adapt_period=p)
    a, b = run(2), run(0)
    for r0, r1 in zip(a, b):
        assert np.array_equal(r0[0]["resident_after"], r1[0]["resident_after"])
        assert r0[0]["capacity"] == 3


# ----------------------------------------------- planted mistakes get caught
class _StatsQuarter(O.AdaptStats):
    def observe(self, layer, n_active, n_hits, capacity, n_experts):
        a_obs = float(n_active) / float(n_experts)
        self.a[layer] = 0.25 * a_obs + 0.75 * self.a[layer] if self.has_a[layer] else a_obs
        self.has_a[layer] = True
        if capacity > 0:
            u_obs = float(n_hits) / float(capacity)
            self.u[layer] = 0.25 * u_obs + 0.75 * self.u[layer] if self.has_u[layer] else u_obs
            self.has_u[layer] = True


def _caps_sum_weight(stats, c_total, E, old):
    st = _stats([x + y for x, y in zip(stats.a, stats.u)], [1.0] * len(stats.a))
    return O.adapt_capacities(st, c_total, E, old)


def _caps_ties_high(stats, c_total, E, old):
    L = len(stats.a)
    rev = _stats(stats.a[::-1], stats.u[::-1])
    return O.adapt_capacities(rev, c_total, E, old[::-1])[::-1]


def _caps_no_ceiling(stats, c_total, E, old):
    return O.adapt_capacities(stats, c_total, 10 ** 9, old)


def _shrink_low_first(resident, S, cap):
    return O.adapt_shrink(resident, np.array([1 << 40], np.uint64) - S, cap)


def test_planted_mistakes_are_caught():
    with pytest.raises(AssertionError):
        check_ema(_StatsQuarter, [(8, 2, 4), (0, 4, 4), (4, 0, 4)], 8, 4)
    with pytest.raises(AssertionError):
        check_capacities_bruteforce(_caps_sum_weight, [0.5, 0.25, 0.125], [0.25, 1.0, 0.5], 5, 8)
    with pytest.raises(AssertionError):
        assert _caps_ties_high(_stats([0.5] * 4, [0.5] * 4), 6, 8, [0] * 4) == [2, 2, 1, 1]
    with pytest.raises(AssertionError):
        check_capacities_bruteforce(_caps_no_ceiling, [1.0, 0.125, 0.125], [1.0, 1.0, 1.0], 6, 4)
    S = np.array([3, 1, 0, 2, 0, 5], np.uint64)
    res = np.array([1, 1, 1, 1, 0, 1], bool)
    with pytest.raises(AssertionError):
        check_shrink_bruteforce(_shrink_low_first, S, res, 2)
