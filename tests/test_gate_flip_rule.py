"""The GPU tests' acceptance rule for a gate that differs from the oracle's
(runs on the CPU): only a one-ulp difference whose exact value sits within the
float64 evaluation's error bound of the fp32 rounding midpoint is accepted,
and the priority numerators and the retained set are then re-judged on the
GPU's gates."""
import mpmath
import numpy as np
import pytest

import gpu_common as G
from oracle import oled_oracle as O


def _ulp_up(v):
    return np.nextafter(np.float32(v), np.float32(np.inf))


def test_identical_gates_need_no_reconciling():
    lg = np.array([[2.0, 1.0, 0.0, -1.0]], np.float32)
    conf = np.array([0.7], np.float32)
    o = O.layer_step(lg, conf, np.zeros(4, bool), 2, 2)
    st = dict(topk_idx=o["idx"], gates=o["gates"].copy())
    assert G.reconcile_gates(st, o, lg, conf, 2, "same") is o


def test_far_from_midpoint_is_rejected():
    lg = np.array([[2.0, 1.0, 0.0, -1.0]], np.float32)
    idx, gates = O.route(lg, 2)
    j = 0
    bumped = _ulp_up(gates[0, j])
    assert not G.accepted_gate_flip(lg[0], idx[0], j, bumped, gates[0, j])
    two = _ulp_up(bumped)
    assert not G.accepted_gate_flip(lg[0], idx[0], j, two, gates[0, j])


def test_at_midpoint_is_accepted_and_rejudged(monkeypatch):
    lg = np.array([[0.5, 0.25, -1.0], [1.0, 0.0, -2.0]], np.float32)
    conf = np.array([0.9, 0.6], np.float32)
    o = O.layer_step(lg, conf, np.zeros(3, bool), 2, 1)
    o["capacity"] = 1
    g_or = o["gates"][0, 1]
    g_gpu = _ulp_up(g_or)
    mid = (mpmath.mpf(float(g_or)) + mpmath.mpf(float(g_gpu))) / 2
    real = G._gate_exact

    def fake(row, sel):        # pretend the exact value sits on the midpoint
        v = real(row, sel)
        if float(row[0]) == 0.5:
            v[1] = mid
        return v

    monkeypatch.setattr(G, "_gate_exact", fake)
    gates = o["gates"].copy()
    gates[0, 1] = g_gpu
    st = dict(topk_idx=o["idx"], gates=gates)
    r = G.reconcile_gates(st, o, lg, conf, 1, "mid")
    assert r is not o and r["gate_flips"] == 1
    S, _ = O.score(o["idx"], gates, conf, 3)
    np.testing.assert_array_equal(r["S"], S)
    np.testing.assert_array_equal(r["resident_after"],
                                  O.retain(S, o["resident_before"], o["miss"], 1))


def test_other_differences_fail():
    lg = np.array([[2.0, 1.0, 0.0]], np.float32)
    conf = np.array([0.5], np.float32)
    o = O.layer_step(lg, conf, np.zeros(3, bool), 2, 2)
    gates = o["gates"].copy()
    gates[0, 0] = _ulp_up(gates[0, 0])
    with pytest.raises(AssertionError):
        G.reconcile_gates(dict(topk_idx=o["idx"], gates=gates), o, lg, conf, 2, "far")
    idx = o["idx"].copy()
    idx[0] = idx[0, ::-1]
    with pytest.raises(AssertionError):
        G.reconcile_gates(dict(topk_idx=idx, gates=o["gates"]), o, lg, conf, 2, "idx")
