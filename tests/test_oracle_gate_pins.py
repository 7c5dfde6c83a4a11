"""Pins of the oracle's gate (O13): the logits against an exact rational sum
of the products, one-hot inputs picking a gate column, and the fp32
accumulation bound holding for float32 sums in several orders. Planted
mistakes fail."""
from fractions import Fraction

import numpy as np
import pytest

from oracle import oled_oracle as O


def check_logits_exact(router_logits, x, wg):
    got = router_logits(x, wg)
    T, H = x.shape
    E = wg.shape[0]
    for t in range(T):
        for e in range(E):
            exact = sum(Fraction(float(x[t, h])) * Fraction(float(wg[e, h])) for h in range(H))
            scale = sum(abs(Fraction(float(x[t, h])) * Fraction(float(wg[e, h]))) for h in range(H))
            assert abs(Fraction(got[t, e]) - exact) <= scale * Fraction(H, 2 ** 52), (t, e)


@pytest.mark.parametrize("seed", range(4))
def test_logits_exact(seed):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((5, 24)).astype(np.float32).astype(np.float64)
    wg = rng.standard_normal((7, 24)).astype(np.float32).astype(np.float64)
    check_logits_exact(O.router_logits, x, wg)


def test_one_hot_rows_pick_gate_columns():
    rng = np.random.default_rng(9)
    wg = rng.standard_normal((6, 16))
    x = np.eye(16)[[3, 0, 15]]
    assert np.array_equal(O.router_logits(x, wg), wg[:, [3, 0, 15]].T)


def test_fp32_bound_holds():
    rng = np.random.default_rng(11)
    x = rng.standard_normal((4, 2048)).astype(np.float32)
    wg = rng.standard_normal((8, 2048)).astype(np.float32)
    ref = O.router_logits(x, wg)
    bound = O.fp32_sum_bound(x, wg)
    prods = x[:, None, :].astype(np.float64) * wg[None, :, :].astype(np.float64)
    for order in (np.arange(2048), np.arange(2048)[::-1], rng.permutation(2048)):
        acc = np.zeros((4, 8), np.float32)
        for h in order:
            acc = (acc + prods[:, :, h].astype(np.float32)).astype(np.float32)
        assert np.all(np.abs(acc.astype(np.float64) - ref) <= bound)
    pair = prods.astype(np.float32).reshape(4, 8, 64, 32).sum(axis=3, dtype=np.float32).sum(
        axis=2, dtype=np.float32)
    assert np.all(np.abs(pair.astype(np.float64) - ref) <= bound)


def test_planted_mistakes_are_caught():
    rng = np.random.default_rng(2)
    x = rng.standard_normal((3, 8))
    wg = rng.standard_normal((4, 8))
    with pytest.raises(AssertionError):
        check_logits_exact(lambda a, b: a @ b[:, ::-1].T, x, wg)
    with pytest.raises(AssertionError):
        check_logits_exact(lambda a, b: (a @ b.T) * (1 + 1e-9), x, wg)
