"""Pins of the oracle's comparison policies (O11): LRU and LFU retention keys
recomputed by brute force from the whole activation history, cross-policy
special cases, the ideal cache bound as an upper bound of every policy, and
the effective transfer ratio recomputed from the resident sets. Planted
mistakes fail."""
import numpy as np
import pytest

from oracle import oled_oracle as O

from test_oracle_pins import check_retain_bruteforce


def _logits(seed, L=2, N=7, T=10, E=8, spread=1.5):
    rng = np.random.default_rng(seed)
    base = rng.standard_normal((L, T, E)) * spread
    lg = np.cumsum(rng.standard_normal((N, L, T, E)) * 0.7, axis=0) + base[None]
    conf = rng.uniform(0, 1, (N, T)).astype(np.float32)
    return lg.astype(np.float32), conf


def _run(seed, policy, C=3, k=2, **kw):
    lg, conf = _logits(seed, **kw)
    N, L, T, E = lg.shape
    return O.run_schedule(lambda l, i: lg[i, l], lambda l, i: conf[i], L, N, E, k, C,
                          policy=policy), E


def brute_keys(steps, l, i, policy, E):
    """The key of every expert at layer l, iteration i, from the history alone."""
    key = []
    for e in range(E):
        if policy == "lru":
            last = [j + 1 for j in range(i + 1) if steps[j][l]["counts"][e] > 0]
            key.append(last[-1] if last else 0)
        else:
            key.append(sum(int(steps[j][l]["counts"][e]) for j in range(i + 1)))
    return key


def check_policy_schedule(steps, policy, E, C):
    for i, row in enumerate(steps):
        for l, st in enumerate(row):
            key = brute_keys(steps, l, i, policy, E)
            assert [int(x) for x in st["key"]] == key, (policy, l, i)
            # the retention itself against brute force over C-subsets
            check_retain_bruteforce(lambda S, r, m, c: O.retain(S, r, m, c),
                                    np.array(key, np.uint64), st["resident_before"], st["miss"], C)
            assert np.array_equal(st["resident_after"],
                                  O.retain(np.array(key, np.uint64), st["resident_before"],
                                           st["miss"], C))


@pytest.mark.parametrize("policy", ["lru", "lfu"])
@pytest.mark.parametrize("seed", range(4))
def test_policy_keys_bruteforce(policy, seed):
    C = 2 + seed % 3
    steps, E = _run(300 + seed, policy, C=C)
    check_policy_schedule(steps, policy, E, C)


def test_first_iteration_special_cases():
    # k = 1 and confidence 1: S = routes * 2^48, so priority and LFU keep the
    # same experts at the first iteration; LRU keeps the lowest ids (all tie)
    rng = np.random.default_rng(5)
    lg = rng.standard_normal((1, 1, 12, 8)).astype(np.float32)
    conf = np.ones((1, 12), np.float32)
    run = lambda pol: O.run_schedule(lambda l, i: lg[i, l], lambda l, i: conf[i], 1, 1, 8, 1, 3,
                                     policy=pol)[0][0]
    pri, lfu, lru = run("priority"), run("lfu"), run("lru")
    assert np.array_equal(pri["S"], pri["counts"].astype(np.uint64) << np.uint64(48))
    assert np.array_equal(pri["resident_after"], lfu["resident_after"])
    act = np.nonzero(lru["active"])[0]
    assert set(np.nonzero(lru["resident_after"])[0]) == set(act[:3])


@pytest.mark.parametrize("policy", ["priority", "lru", "lfu"])
def test_ideal_bound_bounds_every_policy(policy):
    for C in (0, 2, 4, 8):
        steps, E = _run(400 + C, policy, C=C)
        for row in steps:
            for st in row:
                assert st["n_hits"] <= O.ideal_hits(st["n_active"], C)
    assert O.ideal_hits(5, 3) == 3 and O.ideal_hits(2, 3) == 2


def transfer_ratio_from_sets(steps):
    moved = reused = 0
    for l in range(len(steps[0])):
        for i in range(1, len(steps)):
            m = steps[i - 1][l]["miss"]
            kept = m & steps[i][l]["resident_before"]
            moved += int(m.sum())
            reused += int((kept & steps[i][l]["active"]).sum())
    return reused / moved if moved else 0.0


@pytest.mark.parametrize("policy", ["priority", "lru", "lfu"])
def test_effective_transfer_ratio(policy):
    for C in (0, 3, 8):
        steps, E = _run(500 + C, policy, C=C)
        r = O.effective_transfer_ratio(steps)
        assert r == transfer_ratio_from_sets(steps)
        assert 0.0 <= r <= 1.0
        if C == 0:
            assert r == 0.0
        if C == E:   # full residency keeps every transfer: reused = activated again
            moved = sum(int(steps[i][l]["miss"].sum()) for i in range(len(steps) - 1)
                        for l in range(len(steps[0])))
            again = sum(int((steps[i][l]["miss"] & steps[i + 1][l]["active"]).sum())
                        for i in range(len(steps) - 1) for l in range(len(steps[0])))
            assert r == (again / moved if moved else 0.0)


# ----------------------------------------------- planted mistakes get caught
class _FirstUse(O.PolicyHistory):
    def observe(self, counts):
        self.iters += 1
        for e, c in enumerate(counts):
            if c > 0:
                if self.last_use[e] == 0:
                    self.last_use[e] = self.iters
                self.freq[e] += 1   # iterations instead of routes


def test_planted_mistakes_are_caught(monkeypatch):
    monkeypatch.setattr(O, "PolicyHistory", _FirstUse)
    for policy in ("lru", "lfu"):
        steps, E = _run(321, policy, C=3)
        with pytest.raises(AssertionError):
            check_policy_schedule(steps, policy, E, 3)
