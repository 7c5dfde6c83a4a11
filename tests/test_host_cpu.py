"""CPU-only checks of the library: it loads and exports every symbol of the
header, the binding's structures match the header's layout, it validates
arguments before touching a GPU, and the expert packing follows its
documented layout."""
import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

from paper_2609_33385_amd import oled

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "oled.h")


def header_functions():
    text = open(HEADER).read()
    return re.findall(r"^\s*(?:oled_status|void|size_t|const char\s*\*)\s+(\w+)\s*\(", text,
                      re.M)


def test_library_exports_header_symbols():
    names = header_functions()
    assert set(names) == set(oled.EXPORTED), names
    lib = oled.load()
    out = subprocess.run(["nm", "-D", "--defined-only", oled.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = {ln.split()[-1] for ln in out.splitlines() if ln.strip()}
    for n in names:
        assert n in exported, n
        assert getattr(lib, n) is not None


def test_library_targets_gfx950():
    out = subprocess.run(["/opt/rocm/bin/roc-obj-ls", oled.LIB_PATH], capture_output=True,
                         text=True)
    if out.returncode != 0:
        pytest.skip("roc-obj-ls unavailable")
    assert "gfx950" in out.stdout


def _cfg(**kw):
    base = dict(hidden=256, inter=512, n_experts=8, top_k=2, n_layers=1, capacity=4,
                max_tokens=32, dtype=oled.OLED_F32, device=0, profile_ops=0, host_pool=None,
                host_pool_blocks=0, host_block_of=None)
    base.update(kw)
    hbo = np.zeros(base["n_layers"] * base["n_experts"], np.int64)
    c = oled.OledConfig(base["hidden"], base["inter"], base["n_experts"], base["top_k"],
                        base["n_layers"], base["capacity"], base["max_tokens"], base["dtype"],
                        base["device"], base["profile_ops"], base["host_pool"] or 0,
                        base["host_pool_blocks"],
                        hbo.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), 0, 0, 0, 0, 0, 0,
                        0.0, 0.0, 0.0, 0.0)
    return c, hbo


@pytest.mark.parametrize("kw,status", [
    (dict(hidden=0), oled.OLED_ERR_INVALID_ARG),
    (dict(top_k=9), oled.OLED_ERR_INVALID_ARG),
    (dict(dtype=7), oled.OLED_ERR_INVALID_ARG),
    (dict(hidden=200, host_pool=1, host_pool_blocks=1), oled.OLED_ERR_UNSUPPORTED),
    (dict(n_experts=300, top_k=2, host_pool=1, host_pool_blocks=1), oled.OLED_ERR_UNSUPPORTED),
    (dict(max_tokens=70000, host_pool=1, host_pool_blocks=1), oled.OLED_ERR_UNSUPPORTED),
    (dict(capacity=-1), oled.OLED_ERR_INVALID_ARG),
    (dict(), oled.OLED_ERR_INVALID_ARG),  # no host pool
])
def test_create_validates_before_device(kw, status):
    lib = oled.load()
    cfg, _hbo = _cfg(**kw)
    h = ctypes.c_void_p()
    assert lib.oled_create(ctypes.byref(cfg), ctypes.byref(h)) == status
    assert h.value is None
    assert lib.oled_last_error(None)


def test_null_context_calls():
    lib = oled.load()
    assert lib.route_block(None, 0, None, 1, None) == oled.OLED_ERR_INVALID_ARG
    assert lib.apply_misses(None, 0, None, None) == oled.OLED_ERR_INVALID_ARG
    assert lib.moe_forward_cached(None, 0, None, None, None) == oled.OLED_ERR_INVALID_ARG
    assert lib.score_and_retain(None, 0, None, None) == oled.OLED_ERR_INVALID_ARG
    assert lib.oled_reset_cache(None) == oled.OLED_ERR_INVALID_ARG
    lib.oled_destroy(None)


# ------------------------------------------------------- ABI struct layout
ABI_STRUCTS = {
    "oled_config": oled.OledConfig,
    "oled_miss_report": oled.MissReport,
    "oled_stats": oled.Stats,
    "oled_layer_state": oled.LayerState,
    "oled_op_time": oled.OpTime,
}


def test_binding_structs_match_header(tmp_path):
    """The ctypes structures have the header's size and field offsets."""
    lines = ['#include <stddef.h>', '#include <stdio.h>', '#include "oled.h"', 'int main(void) {']
    for cname, py in ABI_STRUCTS.items():
        lines.append(f'  printf("{cname} size %zu\\n", sizeof({cname}));')
        for fname, _ in py._fields_:
            lines.append(f'  printf("{cname} {fname} %zu\\n", offsetof({cname}, {fname}));')
    lines += ["  return 0;", "}"]
    src = tmp_path / "abi.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "abi"
    r = subprocess.run(["gcc", "-std=c99", f"-I{os.path.join(ROOT, 'include')}", str(src), "-o",
                        str(exe)], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    out = subprocess.run([str(exe)], capture_output=True, text=True, check=True).stdout
    got = {}
    for ln in out.splitlines():
        cname, key, val = ln.split()
        got[(cname, key)] = int(val)
    for cname, py in ABI_STRUCTS.items():
        assert got[(cname, "size")] == ctypes.sizeof(py), cname
        for fname, _ in py._fields_:
            assert got[(cname, fname)] == getattr(py, fname).offset, (cname, fname)


def test_create_rejects_bad_copy_mode():
    lib = oled.load()
    cfg, _hbo = _cfg(host_pool=1, host_pool_blocks=1)
    cfg.copy_mode = 5
    h = ctypes.c_void_p()
    assert lib.oled_create(ctypes.byref(cfg), ctypes.byref(h)) == oled.OLED_ERR_INVALID_ARG
    assert b"copy_mode" in lib.oled_last_error(None)


# ------------------------------------------------------------ weight packing
def _pack_ref(w13, w2, H, I, span):
    """Documented packed layout, by reshape/transpose: fragment (q, s) holds
    element (lane = g*16 + r, i) <- row 16q + r, column span*s + V*g + i."""
    V = span // 4

    def frags(M, rows, cols):
        A = M.reshape(rows // 16, 16, cols // span, 4, V).transpose(0, 2, 3, 1, 4)
        return A.reshape(rows // 16, cols // span, 64 * V)

    up = np.stack([frags(w13[:I], I, H), frags(w13[I:], I, H)], axis=2)
    return np.concatenate([up.ravel(), frags(w2, H, I).ravel()])


@pytest.mark.parametrize("dtype,H,I", [("bf16", 256, 128), ("bf16", 128, 384), ("f32", 128, 256)])
def test_pack_expert_layout(dtype, H, I):
    rng = np.random.default_rng(H + I)
    dt = np.uint16 if dtype == "bf16" else np.uint32
    w13 = rng.integers(0, 2 ** 16 if dtype == "bf16" else 2 ** 31, size=(2 * I, H)).astype(dt)
    w2 = rng.integers(0, 2 ** 16 if dtype == "bf16" else 2 ** 31, size=(H, I)).astype(dt)
    out = np.zeros(3 * H * I, dt)
    oled.oled_pack_expert(dtype, H, I, w13 if dtype == "bf16" else w13.view(np.float32),
                          w2 if dtype == "bf16" else w2.view(np.float32),
                          out if dtype == "bf16" else out.view(np.float32))
    ref = _pack_ref(w13, w2, H, I, 32 if dtype == "bf16" else 16)
    assert np.array_equal(out, ref)
    assert sorted(out.tolist()) == sorted(np.concatenate([w13.ravel(), w2.ravel()]).tolist())


def test_pack_expert_errors():
    lib = oled.load()
    a = np.zeros(3 * 128 * 128, np.uint16)
    assert lib.oled_pack_expert(oled.OLED_BF16, 100, 128, a.ctypes.data, a.ctypes.data,
                                a.ctypes.data) == oled.OLED_ERR_UNSUPPORTED
    assert lib.oled_pack_expert(9, 128, 128, a.ctypes.data, a.ctypes.data,
                                a.ctypes.data) == oled.OLED_ERR_INVALID_ARG
    assert lib.oled_pack_expert(oled.OLED_BF16, 128, 128, None, a.ctypes.data,
                                a.ctypes.data) == oled.OLED_ERR_INVALID_ARG


def test_create_rejects_bad_adapt_period():
    lib = oled.load()
    h = ctypes.c_void_p()
    cfg, _hbo = _cfg(host_pool=1, host_pool_blocks=1)
    cfg.adapt_period = -1
    assert lib.oled_create(ctypes.byref(cfg), ctypes.byref(h)) == oled.OLED_ERR_INVALID_ARG
    assert b"adapt_period" in lib.oled_last_error(None)
    cfg, _hbo = _cfg(host_pool=1, host_pool_blocks=1, n_layers=1025)
    cfg.adapt_period = 5
    assert lib.oled_create(ctypes.byref(cfg), ctypes.byref(h)) == oled.OLED_ERR_UNSUPPORTED
    assert h.value is None


def test_create_rejects_bad_policy():
    lib = oled.load()
    h = ctypes.c_void_p()
    cfg, _hbo = _cfg(host_pool=1, host_pool_blocks=1)
    cfg.policy = 3
    assert lib.oled_create(ctypes.byref(cfg), ctypes.byref(h)) == oled.OLED_ERR_INVALID_ARG
    assert b"policy" in lib.oled_last_error(None)


def test_route_noalloc_checks_arguments_before_the_gpu():
    """The allocation-free routing call rejects bad sizes and NULL buffers on
    the host (no device is touched), with the reason in oled_last_error(NULL)."""
    lib = oled.load()
    d = 0x1000    # never dereferenced: every call below fails its host checks
    assert lib.oled_route_noalloc_scratch_bytes() >= 4 * 128 * 256
    cases = [((None, 8, 8, 2), oled.OLED_ERR_INVALID_ARG),
             ((d, 0, 8, 2), oled.OLED_ERR_INVALID_ARG),
             ((d, 8, 8, 9), oled.OLED_ERR_INVALID_ARG),
             ((d, 65536, 8, 2), oled.OLED_ERR_UNSUPPORTED),
             ((d, 8, 257, 2), oled.OLED_ERR_UNSUPPORTED),
             ((d, 8, 64, 17), oled.OLED_ERR_UNSUPPORTED)]
    for (lg, T, E, k), want in cases:
        st = lib.oled_route_noalloc(lg, T, E, k, d, d, d, d, d, d, None, None)
        assert st == want, (T, E, k)
        assert "oled_route_noalloc" in oled.last_error(None)
    assert lib.oled_route_noalloc(d, 8, 8, 2, d, None, d, d, d, d, None, None) == \
        oled.OLED_ERR_INVALID_ARG


def test_batch_calls_check_arguments_before_the_gpu():
    """The batched routing and priority calls reject bad sizes, NULL buffers
    and a short workspace on the host."""
    lib = oled.load()
    d = 0x1000    # never dereferenced: every call below fails its host checks
    ws = lib.oled_route_batch_workspace(4, 3000, 128)
    assert ws >= 4 * 4 * 6 * 128
    assert lib.oled_route_batch_workspace(0, 10, 10) == 0
    rb = lib.oled_route_batch
    assert rb(d, 4, 3000, 128, 8, d, d, d, d, d, d, None, d, ws - 4, None) == \
        oled.OLED_ERR_INVALID_ARG
    assert rb(d, 4, 3000, 128, 8, d, d, d, d, d, d, None, None, ws, None) == \
        oled.OLED_ERR_INVALID_ARG
    assert rb(d, 0, 3000, 128, 8, d, d, d, d, d, d, None, d, ws, None) == oled.OLED_ERR_INVALID_ARG
    assert rb(d, 4, 65536, 128, 8, d, d, d, d, d, d, None, d, 1 << 40, None) == \
        oled.OLED_ERR_UNSUPPORTED
    assert rb(d, 5000, 65535, 128, 8, d, d, d, d, d, d, None, d, 1 << 40, None) == \
        oled.OLED_ERR_UNSUPPORTED
    pb = lib.oled_priority_batch
    assert pb(d, d, None, 4, 30, 16, 2, d, None, None) == oled.OLED_ERR_INVALID_ARG
    assert pb(d, d, d, 4, 30, 16, 17, d, None, None) == oled.OLED_ERR_INVALID_ARG
    assert pb(d, d, d, 4, 65536, 16, 2, d, None, None) == oled.OLED_ERR_UNSUPPORTED
    assert "oled_priority_batch" in oled.last_error(None)
