"""ctypes binding of the C ABI in include/oled.h (argument marshalling only).

Every step of the hot path runs in the HIP library liboled.so; this module
only converts Python/PyTorch arguments into the ABI's pointers and sizes. It
raises if the library is missing: there is no fallback.

Module-level functions carry the ABI's names (route_block, apply_misses,
moe_forward_cached, score_and_retain, ...) and take the context handle first;
`Context` wraps them for convenience.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liboled.so")

OLED_OK = 0
OLED_ERR_INVALID_ARG = 1
OLED_ERR_OUT_OF_MEMORY = 2
OLED_ERR_HIP = 3
OLED_ERR_STATE = 4
OLED_ERR_UNSUPPORTED = 5
STATUS_NAMES = {0: "OK", 1: "INVALID_ARG", 2: "OUT_OF_MEMORY", 3: "HIP", 4: "STATE",
                5: "UNSUPPORTED"}

OLED_F32 = 0
OLED_BF16 = 1
OLED_COPY_SHADER = 0
OLED_COPY_SDMA = 1
COPY_MODES = {"shader": OLED_COPY_SHADER, "sdma": OLED_COPY_SDMA}
POLICIES = {"priority": 0, "lru": 1, "lfu": 2}
PROFILE_ALL = 0x7FF

OP_NAMES = {0: "route_topk", 1: "permute", 2: "ffn_up", 3: "ffn_down", 4: "combine",
            5: "score_retain", 6: "h2d", 7: "ffn_dense_up", 8: "ffn_dense_down",
            9: "layer_adapt", 10: "route_gemm"}
OP_KIND = {v: k for k, v in OP_NAMES.items()}


def profile_mask(*names) -> int:
    """Bitmask of oled_op_kind for oled_config.profile_ops."""
    m = 0
    for n in names:
        m |= 1 << OP_KIND[n]
    return m

EXPORTED = ["oled_create", "oled_destroy", "oled_last_error", "oled_reset_cache", "route_block",
            "route_block_gate",
            "apply_misses", "apply_misses_coop", "moe_forward_cached", "score_and_retain",
            "oled_read_layer_state", "oled_collect_stats", "oled_profile_collect",
            "oled_pack_expert", "oled_host_alloc", "oled_host_free", "oled_coop_dispatch",
            "oled_cpu_ffn", "oled_route_noalloc", "oled_route_noalloc_scratch_bytes",
            "oled_set_fault_injection", "oled_route_batch", "oled_route_batch_workspace",
            "oled_priority_batch"]


class OledConfig(ctypes.Structure):
    _fields_ = [("hidden", ctypes.c_int32), ("inter", ctypes.c_int32),
                ("n_experts", ctypes.c_int32), ("top_k", ctypes.c_int32),
                ("n_layers", ctypes.c_int32), ("capacity", ctypes.c_int32),
                ("max_tokens", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("device", ctypes.c_int32), ("profile_ops", ctypes.c_int32),
                ("host_pool", ctypes.c_void_p), ("host_pool_blocks", ctypes.c_int64),
                ("host_block_of", ctypes.POINTER(ctypes.c_int64)),
                ("copy_mode", ctypes.c_int32), ("adapt_period", ctypes.c_int32),
                ("policy", ctypes.c_int32), ("coop", ctypes.c_int32),
                ("coop_threads", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("coop_t_h2d_us", ctypes.c_double), ("coop_tau_cpu_us", ctypes.c_double),
                ("coop_nbar", ctypes.c_double), ("coop_lambda_us", ctypes.c_double)]


class MissReport(ctypes.Structure):
    _fields_ = [("n_active", ctypes.c_int32), ("n_hits", ctypes.c_int32),
                ("n_misses", ctypes.c_int32), ("n_resident", ctypes.c_int32),
                ("rejected_layer", ctypes.c_int32), ("n_cpu", ctypes.c_int32),
                ("h2d_bytes", ctypes.c_int64)]


class Stats(ctypes.Structure):
    _fields_ = [("layer_iters", ctypes.c_int64), ("n_active", ctypes.c_int64),
                ("n_hits", ctypes.c_int64), ("n_misses", ctypes.c_int64),
                ("n_transferred", ctypes.c_int64), ("h2d_bytes", ctypes.c_int64),
                ("n_bad_blocks", ctypes.c_int64), ("n_prev_transferred", ctypes.c_int64),
                ("n_transfers_reused", ctypes.c_int64), ("n_ideal_hits", ctypes.c_int64),
                ("n_cpu_executed", ctypes.c_int64), ("n_miss_rows", ctypes.c_int64)]

    def as_dict(self) -> dict:
        return {name: getattr(self, name) for name, _ in self._fields_}


class LayerState(ctypes.Structure):
    _fields_ = [("topk_idx", ctypes.c_void_p), ("gates", ctypes.c_void_p),
                ("counts", ctypes.c_void_p), ("offsets", ctypes.c_void_p),
                ("perm", ctypes.c_void_p), ("inv_perm", ctypes.c_void_p),
                ("score_q", ctypes.c_void_p), ("resident_before", ctypes.c_void_p),
                ("resident_after", ctypes.c_void_p), ("slot_of", ctypes.c_void_p),
                ("tokens", ctypes.c_int32), ("n_active", ctypes.c_int32),
                ("n_hits", ctypes.c_int32), ("n_misses", ctypes.c_int32),
                ("capacity", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("retain_key", ctypes.c_void_p), ("prev_transferred", ctypes.c_int32),
                ("reused_transfers", ctypes.c_int32), ("logits", ctypes.c_void_p),
                ("retained", ctypes.c_void_p)]


class OpTime(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("layer", ctypes.c_int32), ("ms", ctypes.c_float),
                ("bytes", ctypes.c_int64), ("flops", ctypes.c_int64),
                ("h2d_bytes", ctypes.c_int64)]


class OledError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


_lib = None


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Loads liboled.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: build it with `python -m paper_2609_33385_amd.build`")
    lib = ctypes.CDLL(path)
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    sig = {
        "oled_create": (i32, [ctypes.POINTER(OledConfig), ctypes.POINTER(vp)]),
        "oled_destroy": (None, [vp]),
        "oled_last_error": (ctypes.c_char_p, [vp]),
        "oled_reset_cache": (i32, [vp]),
        "route_block": (i32, [vp, i32, vp, i32, vp]),
        "route_block_gate": (i32, [vp, i32, vp, vp, i32, vp]),
        "apply_misses": (i32, [vp, i32, vp, ctypes.POINTER(MissReport)]),
        "apply_misses_coop": (i32, [vp, i32, vp, ctypes.POINTER(MissReport)]),
        "oled_coop_dispatch": (i32, [i32, vp, vp, vp, ctypes.c_double, ctypes.c_double,
                                     ctypes.c_double, ctypes.c_double, vp]),
        "oled_cpu_ffn": (i32, [i32, i32, i32, vp, vp, i32, vp, i32]),
        "moe_forward_cached": (i32, [vp, i32, vp, vp, vp]),
        "score_and_retain": (i32, [vp, i32, vp, vp]),
        "oled_read_layer_state": (i32, [vp, i32, ctypes.POINTER(LayerState)]),
        "oled_collect_stats": (i32, [vp, ctypes.POINTER(Stats)]),
        "oled_profile_collect": (i32, [vp, ctypes.POINTER(OpTime), i32, ctypes.POINTER(i32)]),
        "oled_pack_expert": (i32, [i32, i32, i32, vp, vp, vp]),
        "oled_host_alloc": (i32, [i64, ctypes.POINTER(vp)]),
        "oled_host_free": (None, [vp]),
        "oled_route_noalloc": (i32, [vp, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp]),
        "oled_set_fault_injection": (i32, [vp, i32, i32]),
        "oled_route_batch": (i32, [vp, i32, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp,
                                   ctypes.c_size_t, vp]),
        "oled_route_batch_workspace": (ctypes.c_size_t, [i32, i32, i32]),
        "oled_priority_batch": (i32, [vp, vp, vp, i32, i32, i32, i32, vp, vp, vp]),
        "oled_route_noalloc_scratch_bytes": (ctypes.c_size_t, []),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _ptr(x) -> int | None:
    """Device/host address of a torch tensor, numpy array, int or None."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if hasattr(x, "data_ptr"):
        return x.data_ptr()
    if isinstance(x, np.ndarray):
        return x.ctypes.data
    raise TypeError(f"cannot take the address of {type(x)}")


def _stream(s) -> int | None:
    if s is None:
        return None
    if isinstance(s, int):
        return s
    return s.cuda_stream  # torch.cuda.Stream


def last_error(ctx) -> str:
    return load().oled_last_error(ctx).decode()


def _check(ctx, status: int):
    if status != OLED_OK:
        raise OledError(status, last_error(ctx))


# ------------------------------------------------------------ ABI functions
def oled_create(cfg: OledConfig) -> int:
    lib = load()
    h = ctypes.c_void_p()
    st = lib.oled_create(ctypes.byref(cfg), ctypes.byref(h))
    if st != OLED_OK:
        raise OledError(st, lib.oled_last_error(None).decode())
    return h.value


def oled_destroy(ctx) -> None:
    load().oled_destroy(ctx)


def oled_reset_cache(ctx) -> None:
    _check(ctx, load().oled_reset_cache(ctx))


def route_block(ctx, layer: int, logits, T: int, stream=None) -> int:
    return load().route_block(ctx, layer, _ptr(logits), T, _stream(stream))


def route_block_gate(ctx, layer: int, x, w_gate, T: int, stream=None) -> int:
    return load().route_block_gate(ctx, layer, _ptr(x), _ptr(w_gate), T, _stream(stream))


def apply_misses(ctx, layer: int, copy_stream=None, report: MissReport | None = None) -> int:
    return load().apply_misses(ctx, layer, _stream(copy_stream),
                               ctypes.byref(report) if report is not None else None)


def apply_misses_coop(ctx, layer: int, conf, report: MissReport | None = None) -> int:
    return load().apply_misses_coop(ctx, layer, _ptr(conf),
                                    ctypes.byref(report) if report is not None else None)


def oled_coop_dispatch(miss: np.ndarray, n_tok: np.ndarray, score: np.ndarray, t_h2d_us: float,
                       tau_cpu_us: float, nbar: float, lambda_us: float) -> np.ndarray:
    """The library's dispatch of the misses (transfer mask, bool [E])."""
    miss = np.ascontiguousarray(miss, dtype=np.uint8)
    n_tok = np.ascontiguousarray(n_tok, dtype=np.int32)
    score = np.ascontiguousarray(score, dtype=np.uint64)
    out = np.zeros(miss.size, np.uint8)
    st = load().oled_coop_dispatch(miss.size, miss.ctypes.data, n_tok.ctypes.data,
                                   score.ctypes.data, t_h2d_us, tau_cpu_us, nbar, lambda_us,
                                   out.ctypes.data)
    if st != OLED_OK:
        raise OledError(st, "oled_coop_dispatch")
    return out.astype(bool)


def oled_cpu_ffn(dtype: str, hidden: int, inter: int, block: np.ndarray, x: np.ndarray,
                 threads: int = 1) -> np.ndarray:
    """One packed expert's SwiGLU on the host CPU: x [n][H] (float32, or bf16
    bits) -> float32 [n][H]."""
    block = np.ascontiguousarray(block)
    x = np.ascontiguousarray(x)
    n = x.shape[0]
    out = np.zeros((n, hidden), np.float32)
    st = load().oled_cpu_ffn(OLED_F32 if dtype == "f32" else OLED_BF16, hidden, inter,
                             block.ctypes.data, x.ctypes.data, n, out.ctypes.data, threads)
    if st != OLED_OK:
        raise OledError(st, "oled_cpu_ffn")
    return out


def oled_route_noalloc(logits, T: int, E: int, k: int, topk_idx, gates, counts, offsets, perm,
                       inv_perm, nonfinite=None, stream=None) -> int:
    """Routing and permutation without a context (device tensors in, device
    tensors out); returns the status."""
    return load().oled_route_noalloc(_ptr(logits), T, E, k, _ptr(topk_idx), _ptr(gates),
                                     _ptr(counts), _ptr(offsets), _ptr(perm), _ptr(inv_perm),
                                     _ptr(nonfinite), _stream(stream))


def oled_route_batch(logits, B: int, T: int, E: int, k: int, topk_idx, gates, counts, offsets,
                     perm, inv_perm, nonfinite, workspace, stream=None) -> int:
    """Routing and permutation of B independent blocks (device tensors);
    workspace: a device tensor of at least oled_route_batch_workspace(B, T, E)
    bytes. Returns the status."""
    nbytes = workspace.numel() * workspace.element_size()
    return load().oled_route_batch(_ptr(logits), B, T, E, k, _ptr(topk_idx), _ptr(gates),
                                   _ptr(counts), _ptr(offsets), _ptr(perm), _ptr(inv_perm),
                                   _ptr(nonfinite), _ptr(workspace), nbytes, _stream(stream))


def oled_route_batch_workspace(B: int, T: int, E: int) -> int:
    return load().oled_route_batch_workspace(B, T, E)


def oled_priority_batch(topk_idx, gates, conf, B: int, T: int, E: int, k: int, score_q,
                        bad_conf=None, stream=None) -> int:
    """Priority numerators of B independent blocks (device tensors); returns
    the status."""
    return load().oled_priority_batch(_ptr(topk_idx), _ptr(gates), _ptr(conf), B, T, E, k,
                                      _ptr(score_q), _ptr(bad_conf), _stream(stream))


def moe_forward_cached(ctx, layer: int, x, y, stream=None) -> int:
    return load().moe_forward_cached(ctx, layer, _ptr(x), _ptr(y), _stream(stream))


def score_and_retain(ctx, layer: int, conf, stream=None) -> int:
    return load().score_and_retain(ctx, layer, _ptr(conf), _stream(stream))


def oled_read_layer_state(ctx, layer: int, state: LayerState) -> int:
    return load().oled_read_layer_state(ctx, layer, ctypes.byref(state))


def oled_collect_stats(ctx) -> dict:
    st = Stats()
    _check(ctx, load().oled_collect_stats(ctx, ctypes.byref(st)))
    return st.as_dict()


def oled_profile_collect(ctx, cap: int = 1 << 16):
    """[(op name, layer, ms, bytes, flops, h2d_bytes)] since the last collection."""
    arr = (OpTime * cap)()
    n = ctypes.c_int32()
    _check(ctx, load().oled_profile_collect(ctx, arr, cap, ctypes.byref(n)))
    return [(OP_NAMES[arr[i].kind], arr[i].layer, arr[i].ms, arr[i].bytes, arr[i].flops,
             arr[i].h2d_bytes) for i in range(n.value)]


def oled_pack_expert(dtype: str, hidden: int, inter: int, w13: np.ndarray, w2: np.ndarray,
                     out: np.ndarray) -> None:
    """Packs logical w13 [2I][H] and w2 [H][I] (float32 or bf16 bits) into `out`."""
    w13 = np.ascontiguousarray(w13)
    w2 = np.ascontiguousarray(w2)
    assert out.flags.c_contiguous and out.size == 3 * hidden * inter
    st = load().oled_pack_expert(OLED_F32 if dtype == "f32" else OLED_BF16, hidden, inter,
                                 w13.ctypes.data, w2.ctypes.data, out.ctypes.data)
    if st != OLED_OK:
        raise OledError(st, "oled_pack_expert")


def oled_host_alloc(nbytes: int) -> int:
    p = ctypes.c_void_p()
    st = load().oled_host_alloc(nbytes, ctypes.byref(p))
    if st != OLED_OK:
        raise OledError(st, f"pinned host allocation of {nbytes} bytes failed")
    return p.value


def oled_host_free(ptr: int) -> None:
    load().oled_host_free(ptr)


# ---------------------------------------------------------------- helpers
class PinnedPool:
    """Pinned host expert pool of n_blocks blocks of block_bytes (oled_host_alloc)."""

    def __init__(self, n_blocks: int, block_bytes: int):
        self.n_blocks, self.block_bytes = n_blocks, block_bytes
        self.ptr = oled_host_alloc(n_blocks * block_bytes)

    def view(self, dtype=np.uint8) -> np.ndarray:
        buf = (ctypes.c_char * (self.n_blocks * self.block_bytes)).from_address(self.ptr)
        return np.frombuffer(buf, dtype=dtype)

    def block(self, b: int, dtype) -> np.ndarray:
        n = self.block_bytes // np.dtype(dtype).itemsize
        return self.view(dtype)[b * n:(b + 1) * n]

    def free(self):
        if self.ptr:
            oled_host_free(self.ptr)
            self.ptr = 0

    def __del__(self):
        try:
            self.free()
        except Exception:
            pass


class Context:
    """One layer stack with its expert caches (wraps the ABI functions)."""

    def __init__(self, hidden, inter, n_experts, top_k, n_layers, capacity, max_tokens,
                 dtype: str, host_pool: int, host_pool_blocks: int, host_block_of,
                 device: int = 0, profile_ops: int = 0, copy_mode: str = "shader",
                 adapt_period: int = 0, policy: str = "priority", coop: dict | None = None):
        """coop: None, or dict(threads, t_h2d_us, tau_cpu_us, nbar, lambda_us) for the
        cooperative compensation (apply_misses_coop)."""
        self._hbo = np.ascontiguousarray(host_block_of, dtype=np.int64)
        cfg = OledConfig(hidden, inter, n_experts, top_k, n_layers, capacity, max_tokens,
                         OLED_F32 if dtype == "f32" else OLED_BF16, device,
                         profile_ops, host_pool, host_pool_blocks,
                         self._hbo.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)),
                         COPY_MODES[copy_mode], adapt_period, POLICIES[policy],
                         1 if coop else 0, int(coop["threads"]) if coop else 0, 0,
                         float(coop["t_h2d_us"]) if coop else 0.0,
                         float(coop["tau_cpu_us"]) if coop else 0.0,
                         float(coop["nbar"]) if coop else 0.0,
                         float(coop["lambda_us"]) if coop else 0.0)
        self.coop = bool(coop)
        self.E, self.k, self.L, self.C, self.Tmax = n_experts, top_k, n_layers, capacity, max_tokens
        self.ctx = oled_create(cfg)

    def close(self):
        if self.ctx:
            oled_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def reset_cache(self):
        oled_reset_cache(self.ctx)

    def set_fault_injection(self, copy_fail_at: int = 0, wait_deadline_ms: int = 0):
        _check(self.ctx, load().oled_set_fault_injection(self.ctx, copy_fail_at, wait_deadline_ms))

    def route_block(self, layer, logits, T, stream=None):
        _check(self.ctx, route_block(self.ctx, layer, logits, T, stream))

    def route_block_gate(self, layer, x, w_gate, T, stream=None):
        _check(self.ctx, route_block_gate(self.ctx, layer, x, w_gate, T, stream))

    def apply_misses(self, layer, copy_stream=None, report: bool = True) -> MissReport | None:
        """With report=False nothing waits for the device (shader transfer)."""
        rep = MissReport() if report else None
        _check(self.ctx, apply_misses(self.ctx, layer, copy_stream, rep))
        return rep

    def apply_misses_coop(self, layer, conf, report: bool = True) -> MissReport | None:
        rep = MissReport() if report else None
        _check(self.ctx, apply_misses_coop(self.ctx, layer, conf, rep))
        return rep

    def moe_forward_cached(self, layer, x, y, stream=None):
        _check(self.ctx, moe_forward_cached(self.ctx, layer, x, y, stream))

    def score_and_retain(self, layer, conf, stream=None):
        _check(self.ctx, score_and_retain(self.ctx, layer, conf, stream))

    def read_layer_state(self, layer, T=None) -> dict:
        E, k = self.E, self.k
        R = (T if T is not None else self.Tmax) * k
        out = dict(topk_idx=np.zeros(R, np.int32), gates=np.zeros(R, np.float32),
                   counts=np.zeros(E, np.int32), offsets=np.zeros(E + 1, np.int32),
                   perm=np.zeros(R, np.int32), inv_perm=np.zeros(R, np.int32),
                   score_q=np.zeros(E, np.uint64), resident_before=np.zeros(E, np.uint8),
                   resident_after=np.zeros(E, np.uint8), slot_of=np.zeros(E, np.int32))
        rkey = np.zeros(E, np.uint64)
        lgt = np.full(R * E // k, np.nan, np.float32)
        kept = np.zeros(E, np.uint8)
        st = LayerState(*[a.ctypes.data for a in out.values()], 0, 0, 0, 0, 0, 0,
                        rkey.ctypes.data, 0, 0, lgt.ctypes.data, kept.ctypes.data)
        status = oled_read_layer_state(self.ctx, layer, st)
        if status not in (OLED_OK, OLED_ERR_INVALID_ARG):
            _check(self.ctx, status)
        Tn = st.tokens
        for key in ("topk_idx", "gates", "perm", "inv_perm"):
            out[key] = out[key][: Tn * k]
        out["topk_idx"] = out["topk_idx"].reshape(Tn, k)
        out["gates"] = out["gates"].reshape(Tn, k)
        out.update(tokens=Tn, n_active=st.n_active, n_hits=st.n_hits, n_misses=st.n_misses,
                   capacity=st.capacity, retain_key=rkey, prev_transferred=st.prev_transferred,
                   logits=lgt[: Tn * E].reshape(Tn, E),
                   reused_transfers=st.reused_transfers, retained=kept.astype(bool),
                   rejected=(status == OLED_ERR_INVALID_ARG))
        out["resident_before"] = out["resident_before"].astype(bool)
        out["resident_after"] = out["resident_after"].astype(bool)
        return out

    def collect_stats(self) -> dict:
        return oled_collect_stats(self.ctx)

    def profile_collect(self):
        return oled_profile_collect(self.ctx)
