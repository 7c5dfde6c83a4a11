"""CPU-only checks of the cooperative compensation's host code in the library:
the CPU expert kernels against the oracle's SwiGLU (from the same packed
blocks the GPU reads), the dispatch against the oracle's two-stage heuristic
(bit-exact transfer sets over float64 decisions), and argument validation."""
import ctypes

import numpy as np
import pytest

from oracle import oled_oracle as O
from paper_2609_33385_amd import oled
from paper_2609_33385_amd import workload as W

from test_host_cpu import _cfg


def _rel(a, b):
    return float(np.linalg.norm(a - b) / np.linalg.norm(b))


@pytest.mark.parametrize("isa", ["auto", "avx2"])
@pytest.mark.parametrize("dtype,H,I,n,threads", [("bf16", 256, 512, 1, 1), ("bf16", 512, 256, 13, 4),
                                                 ("bf16", 2048, 1024, 3, 8), ("bf16", 256, 256, 29, 3),
                                                 ("f32", 256, 128, 7, 3), ("f32", 128, 384, 20, 1)])
def test_cpu_ffn_matches_oracle(dtype, H, I, n, threads, isa, monkeypatch):
    """Both bf16 kernels: AVX-512 BF16 dot products where the CPU has them
    ("auto"), and the AVX2 kernels (forced)."""
    if isa == "avx2":
        monkeypatch.setenv("OLED_CPU_FFN_AVX2", "1")
    else:
        monkeypatch.delenv("OLED_CPU_FFN_AVX2", raising=False)
    w = W.WORKLOADS[1].replace(wid=340, dtype=dtype, hidden=H, inter=I)
    raw = W.expert_block(w, 0, 3)
    w13, w2 = W.split_expert(w, raw)
    packed = np.zeros(3 * H * I, raw.dtype)
    oled.oled_pack_expert(dtype, H, I, w13, w2, packed)
    x = W.activations(w.replace(batch=1, block=n), 0, 0, 0, 1)
    got = oled.oled_cpu_ffn(dtype, H, I, packed, x, threads).astype(np.float64)
    f13, f2 = W.split_expert(w, O.decode(raw))
    want = O.expert_ffn(O.decode(x), f13, f2)
    err = _rel(got, want)
    assert err <= (2e-2 if dtype == "bf16" else 1e-5), err
    # the thread count does not change the result
    again = oled.oled_cpu_ffn(dtype, H, I, packed, x, 1 if threads > 1 else 2)
    assert np.array_equal(again, got.astype(np.float32))


def _case(rng, E):
    miss = rng.uniform(0, 1, E) < rng.uniform(0.1, 0.9)
    n_tok = np.where(miss, rng.integers(1, 40, E), rng.integers(0, 5, E)).astype(np.int32)
    # numerators on the scale of floor(g c 2^48) sums, ties now and then
    S = (rng.integers(0, 50, E).astype(np.uint64) * np.uint64(1 << 44)
         + rng.integers(0, 1 << 20, E).astype(np.uint64) * (rng.uniform(0, 1, E) < 0.5))
    S[n_tok == 0] = 0
    return miss, n_tok, S


@pytest.mark.parametrize("seed", range(40))
def test_dispatch_matches_oracle(seed):
    rng = np.random.default_rng(seed)
    E = int(rng.choice([8, 64, 128, 256]))
    miss, n_tok, S = _case(rng, E)
    t = float(rng.uniform(20, 400))
    tau = float(rng.choice([0.0, rng.uniform(0.5, 40)]))
    nbar = float(rng.uniform(0, 30))
    lam = float(rng.choice([0.0, rng.uniform(1, 50), rng.uniform(100, 5000), 1e12]))
    got = oled.oled_coop_dispatch(miss, n_tok, S, t, tau, nbar, lam)
    want = O.coop_dispatch(miss, n_tok, S, t, tau, nbar, lam)
    assert np.array_equal(got, want)


def test_dispatch_rejects_bad_arguments():
    lib = oled.load()
    a = np.zeros(8, np.uint8)
    i = np.zeros(8, np.int32)
    s = np.zeros(8, np.uint64)
    o = np.zeros(8, np.uint8)
    assert lib.oled_coop_dispatch(0, a.ctypes.data, i.ctypes.data, s.ctypes.data, 1.0, 1.0, 1.0,
                                  1.0, o.ctypes.data) == oled.OLED_ERR_INVALID_ARG
    assert lib.oled_coop_dispatch(8, a.ctypes.data, i.ctypes.data, s.ctypes.data, -1.0, 1.0, 1.0,
                                  1.0, o.ctypes.data) == oled.OLED_ERR_INVALID_ARG
    assert lib.oled_coop_dispatch(8, None, i.ctypes.data, s.ctypes.data, 1.0, 1.0, 1.0, 1.0,
                                  o.ctypes.data) == oled.OLED_ERR_INVALID_ARG


def test_create_validates_coop_fields():
    lib = oled.load()
    h = ctypes.c_void_p()
    cfg, _hbo = _cfg(host_pool=1, host_pool_blocks=1)
    cfg.coop, cfg.coop_threads = 1, 0
    assert lib.oled_create(ctypes.byref(cfg), ctypes.byref(h)) == oled.OLED_ERR_INVALID_ARG
    cfg.coop_threads, cfg.coop_tau_cpu_us = 4, -2.0
    assert lib.oled_create(ctypes.byref(cfg), ctypes.byref(h)) == oled.OLED_ERR_INVALID_ARG
    cfg.coop_tau_cpu_us, cfg.copy_mode = 3.0, oled.OLED_COPY_SDMA
    assert lib.oled_create(ctypes.byref(cfg), ctypes.byref(h)) == oled.OLED_ERR_UNSUPPORTED
    cfg.copy_mode, cfg.coop = 0, 2
    assert lib.oled_create(ctypes.byref(cfg), ctypes.byref(h)) == oled.OLED_ERR_INVALID_ARG
    assert h.value is None
