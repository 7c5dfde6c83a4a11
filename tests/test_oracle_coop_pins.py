"""Pins of the oracle's cooperative compensation (O12): the split rho in
closed form and at its limits, the transfer count, stage 2 ending in a local
optimum of J (checked over every single swap), the global optimum by brute
force where the objective is load-only, the priority-only limit, monotone
improvement over stage 1, and schedule invariants (CPU-executed experts never
enter the cache). Planted mistakes fail."""
import itertools

import numpy as np
import pytest

from oracle import oled_oracle as O


def _case(seed, E=10, p_miss=0.6):
    rng = np.random.default_rng(seed)
    miss = rng.uniform(0, 1, E) < p_miss
    n_tok = np.where(miss | (rng.uniform(0, 1, E) < 0.5), rng.integers(1, 20, E), 0)
    n_tok[miss & (n_tok == 0)] = 1
    S = (rng.integers(0, 1000, E) * (n_tok > 0)).astype(np.uint64) << np.uint64(30)
    return miss, n_tok, S


def _J(G, miss, n_tok, S, t, tau, lam):
    misses = [e for e in range(len(miss)) if miss[e]]
    return O.coop_objective(set(G), misses, n_tok, S, int(sum(int(x) for x in S)), t, tau, lam)


def check_dispatch(dispatch, miss, n_tok, S, t, tau, nbar, lam):
    G = dispatch(miss, n_tok, S, t, tau, nbar, lam)
    misses = [e for e in range(len(miss)) if miss[e]]
    gset = [e for e in range(len(miss)) if G[e]]
    assert not np.any(G & ~miss)
    rho = O.coop_rho(t, tau, nbar)
    assert len(gset) == int(np.floor(rho * len(misses) + 0.5))
    J = _J(gset, miss, n_tok, S, t, tau, lam)
    for g in gset:          # no single swap lowers J
        for c in misses:
            if c in gset:
                continue
            Gs = [e for e in gset if e != g] + [c]
            assert _J(Gs, miss, n_tok, S, t, tau, lam) >= J, (g, c)
    first = sorted(misses, key=lambda e: (-int(S[e]), e))[:len(gset)]
    assert J <= _J(first, miss, n_tok, S, t, tau, lam)
    return gset, J


def test_rho_closed_form_and_limits():
    assert O.coop_rho(100.0, 5.0, 20.0) == 0.5
    assert O.coop_rho(300.0, 10.0, 10.0) == 0.25
    assert O.coop_rho(0.0, 3.0, 4.0) == 1.0 and O.coop_rho(50.0, 0.0, 4.0) == 0.0
    miss, n_tok, S = _case(1)
    assert not O.coop_dispatch(miss, n_tok, S, 50.0, 0.0, 8.0, 1.0).any()       # CPU is free
    assert np.array_equal(O.coop_dispatch(miss, n_tok, S, 0.0, 3.0, 8.0, 1.0), miss)


@pytest.mark.parametrize("seed", range(30))
def test_dispatch_local_optimum(seed):
    miss, n_tok, S = _case(seed)
    rng = np.random.default_rng(1000 + seed)
    t, tau, nbar = float(rng.uniform(50, 300)), float(rng.uniform(2, 30)), float(rng.uniform(2, 20))
    lam = float(rng.choice([0.0, 10.0, 100.0, 1000.0]))
    check_dispatch(O.coop_dispatch, miss, n_tok, S, t, tau, nbar, lam)


@pytest.mark.parametrize("seed", range(15))
def test_dispatch_load_only_is_globally_optimal(seed):
    miss, n_tok, S = _case(200 + seed, E=9)
    t, tau, nbar = 40.0, 9.0, 6.0
    gset, J = check_dispatch(O.coop_dispatch, miss, n_tok, S, t, tau, nbar, 0.0)
    misses = [e for e in range(len(miss)) if miss[e]]
    best = min(_J(G, miss, n_tok, S, t, tau, 0.0) for G in itertools.combinations(misses, len(gset)))
    assert J == best


def test_dispatch_priority_only_limit():
    # lambda so large that only the transferred priority mass matters: stage 1 stands
    for seed in range(10):
        miss, n_tok, S = _case(300 + seed)
        G = O.coop_dispatch(miss, n_tok, S, 100.0, 10.0, 10.0, 1e15)
        misses = [e for e in range(len(miss)) if miss[e]]
        n_g = int(G.sum())
        top = sorted(misses, key=lambda e: (-int(S[e]), e))[:n_g]
        assert set(np.nonzero(G)[0]) == set(top)


def test_coop_schedule_invariants():
    rng = np.random.default_rng(7)
    L, N, T, E, k, C = 2, 6, 12, 8, 2, 3
    lg = (np.cumsum(rng.standard_normal((N, L, T, E)) * 0.8, axis=0)
          + rng.standard_normal((L, T, E)) * 1.5).astype(np.float32)
    conf = rng.uniform(0, 1, (N, T)).astype(np.float32)
    steps = O.run_coop_schedule(lambda l, i: lg[i, l], lambda l, i: conf[i], L, N, E, k, C,
                                60.0, 8.0, 5.0, 20.0)
    some_cpu = False
    for row in steps:
        for st in row:
            R0, R1, A = st["resident_before"], st["resident_after"], st["active"]
            assert not np.any(st["transfer"] & st["cpu"])
            assert np.array_equal(st["transfer"] | st["cpu"], st["miss"])
            assert not np.any(R1 & st["cpu"])                 # CPU-executed experts stay out
            assert not np.any(R1 & ~(R0 | st["transfer"]))    # R' within R u G
            assert R1.sum() == min(C, (R0 | st["transfer"]).sum())
            some_cpu |= bool(st["cpu"].any())
    assert some_cpu


# ----------------------------------------------- planted mistakes get caught
def _floor_split(miss, n_tok, S, t, tau, nbar, lam):
    rho = O.coop_rho(t, tau, nbar)
    misses = [e for e in range(len(miss)) if miss[e]]
    n_g = int(np.floor(rho * len(misses)))
    G = np.zeros(len(miss), bool)
    for e in sorted(misses, key=lambda e: (-int(S[e]), e))[:n_g]:
        G[e] = True
    return G


def _low_priority_first(miss, n_tok, S, t, tau, nbar, lam):
    return O.coop_dispatch(miss, n_tok, np.uint64(1 << 50) - S, t, tau, nbar, lam)


def test_planted_mistakes_are_caught():
    miss = np.array([1, 1, 1, 1, 1, 0, 0], bool)
    n_tok = np.array([9, 1, 5, 2, 7, 3, 0])
    S = np.array([50, 900, 10, 400, 30, 5, 0], np.uint64) << np.uint64(30)
    args = (120.0, 10.0, 12.0, 1e15)    # rho = 0.5: 2.5 of 5 round up to 3
    check_dispatch(O.coop_dispatch, miss, n_tok, S, *args)
    with pytest.raises(AssertionError):
        check_dispatch(_floor_split, miss, n_tok, S, *args)
    with pytest.raises(AssertionError):
        check_dispatch(_low_priority_first, miss, n_tok, S, *args)
    # load-only: stage 1 alone (no swaps) is not a local optimum here
    with pytest.raises(AssertionError):
        check_dispatch(_floor_split, miss, n_tok, S, 40.0, 9.0, 4.0, 0.0)
