"""Python binding of the C ABI in ``include/wisp.h`` (``libwisp.so``): argument marshalling only.

Every step of the paged MoE layer runs in the library's HIP kernels and host pager; this module
converts arguments, checks status codes and raises on error.  It loads the in-tree
``libwisp.so`` and fails loudly if it is missing.  Device memory and streams come from PyTorch.

``DecodeRun`` wires one workload together (context, pinned masters filled by the seeded input
generator, router weights and hidden states on the device) for tests, the smoke check and the
benchmark.
"""
from __future__ import annotations

import ctypes
import os
import time

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libwisp.so")

OK, E_INVAL, E_NOMEM, E_HIP, E_NOT_RESIDENT, E_STATE = 0, -1, -2, -3, -4, -5
STATUS_NAMES = {0: "OK", -1: "E_INVAL", -2: "E_NOMEM", -3: "E_HIP", -4: "E_NOT_RESIDENT", -5: "E_STATE"}
F32, BF16, FP8 = 0, 1, 2
PAGER_HOST, PAGER_DEVICE = 0, 1
LINK_COPY_ENGINE, LINK_CUS = 0, 1
OFFLOAD_BULK, OFFLOAD_ZERO_COPY = 0, 1
PREFETCH_OFF, PREFETCH_PREDICTOR, PREFETCH_HINTS = 0, 1, 2
(K_ROUTER_LOGITS, K_ROUTER_SELECT, K_FFN_GATEUP, K_FFN_DOWN, K_COMBINE, K_H2D_FILL, K_GROUPED_GATEUP,
 K_GROUPED_DOWN, K_PERMUTE, K_DOWN_COMBINE) = range(10)
KERNEL_CLASS_NAMES = ["router_logits", "router_select", "ffn_gateup", "ffn_down", "combine", "h2d_fill",
                      "grouped_gateup", "grouped_down", "permute", "down_combine"]


class WispError(RuntimeError):
    def __init__(self, status, func, msg):
        super().__init__(f"{func} -> {STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


class ModelDesc(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "n_layers", "d_model", "d_ff", "n_experts", "top_k", "n_groups", "topk_groups", "has_shared", "route",
        "w_dtype", "x_dtype", "max_tokens", "pageable_masters")]


class PageStats(ctypes.Structure):
    _fields_ = [("hits", ctypes.c_uint32), ("misses", ctypes.c_uint32), ("chunks", ctypes.c_uint32),
                ("steps", ctypes.c_uint32), ("h2d_bytes", ctypes.c_uint64)]

    def as_dict(self):
        return dict(hits=self.hits, misses=self.misses, chunks=self.chunks, steps=self.steps,
                    h2d_bytes=self.h2d_bytes)


class MvwsaProblem(ctypes.Structure):
    _fields_ = [("budget_bytes", ctypes.c_uint64), ("expert_set_bytes", ctypes.c_uint64),
                ("kv_block_bytes", ctypes.c_uint64), ("kv_min_blocks", ctypes.c_int64), ("c_exp", ctypes.c_double),
                ("c_kv", ctypes.c_double), ("n_experts", ctypes.c_int32), ("kv_curve_len", ctypes.c_int64)]


class MvwsaSplit(ctypes.Structure):
    _fields_ = [("cap", ctypes.c_int32), ("kv_blocks", ctypes.c_int64), ("kv_bytes", ctypes.c_uint64),
                ("f", ctypes.c_double), ("latency", ctypes.c_double), ("floor_binding", ctypes.c_int32)]


class ResizeLaw(ctypes.Structure):
    _fields_ = [("budget_bytes", ctypes.c_uint64), ("expert_set_bytes", ctypes.c_uint64),
                ("kv_block_bytes", ctypes.c_uint64), ("kv_min_blocks", ctypes.c_int64), ("headroom", ctypes.c_double),
                ("cap_min", ctypes.c_int32), ("cap_max", ctypes.c_int32), ("dead_zone", ctypes.c_int32)]


_lib = None
_P = ctypes.c_void_p
_I = ctypes.c_int32
_U64 = ctypes.c_uint64

# (name, argtypes) for every function of include/*.h
_SIGS = {
    "wisp_expert_bytes": [ctypes.POINTER(ModelDesc), ctypes.POINTER(_U64)],
    "wisp_create": [ctypes.POINTER(ModelDesc), ctypes.POINTER(_P)],
    "wisp_destroy": [_P],
    "wisp_expert_host_ptr": [_P, _I, _I, ctypes.POINTER(_P), ctypes.POINTER(_U64)],
    "wisp_masters_ready": [_P],
    "wisp_router_weights": [_P, _I, _P],
    "wisp_set_budget": [_P, _U64, ctypes.POINTER(_I)],
    "wisp_preload": [_P],
    "wisp_set_pager": [_P, _I],
    "wisp_set_fusion": [_P, _I],
    "wisp_route_topk": [_P, _I, _P, _I, _P, _P, _P, _P],
    "wisp_page_in": [_P, _I, _P, _I, ctypes.POINTER(PageStats)],
    "wisp_moe_forward": [_P, _I, _P, _I, _P, _P, _P, ctypes.POINTER(PageStats)],
    "wisp_decode_step": [_P, _P, _I, _P, _P, _P, _P, _P],
    "wisp_offload_begin": [_P, _U64, _I, ctypes.POINTER(_I)],
    "wisp_offload_step": [_P, _P, _I, _P, _P, _P, _P],
    "wisp_offload_end": [_P],
    "wisp_get_desc": [_P, ctypes.POINTER(ModelDesc)],
    "wisp_miss_curve": [_P, _I, _I, _I, _P, _P],
    "wisp_mvwsa_configure": [ctypes.POINTER(MvwsaProblem), _P, _P, ctypes.POINTER(MvwsaSplit)],
    "wisp_resize_target": [ctypes.POINTER(ResizeLaw), ctypes.c_int64, _I, ctypes.POINTER(_I),
                           ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(_I)],
    "wisp_kv_pool_create": [ctypes.c_uint64, ctypes.c_int64, ctypes.POINTER(_P)],
    "wisp_kv_pool_blocks": [_P, ctypes.POINTER(ctypes.c_int64)],
    "wisp_kv_pool_resize": [_P, ctypes.c_int64],
    "wisp_kv_pool_destroy": [_P],
    "wisp_dual_resize": [_P, _P, _I, ctypes.c_int64],
    "wisp_controller_create": [ctypes.POINTER(ResizeLaw), _I, ctypes.c_int64, ctypes.POINTER(_P)],
    "wisp_controller_observe": [_P, ctypes.c_int64],
    "wisp_controller_barrier": [_P, _P, _P, ctypes.POINTER(_I), ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(_I),
                                ctypes.POINTER(ctypes.c_int64)],
    "wisp_controller_destroy": [_P],
    "wisp_get_stats": [_P, _I, ctypes.POINTER(PageStats)],
    "wisp_reset_stats": [_P],
    "wisp_get_cap": [_P, ctypes.POINTER(_I)],
    "wisp_slot_of": [_P, _I, _I, ctypes.POINTER(_I)],
    "wisp_expert_in_slot": [_P, _I, _I, ctypes.POINTER(_I)],
    "wisp_read_slot": [_P, _I, _I, _P],
    "wisp_set_profiling": [_P, _I],
    "wisp_kernel_times": [_P, _I, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(_U64), ctypes.POINTER(_U64),
                          ctypes.POINTER(_U64)],
    "wisp_reset_kernel_times": [_P],
    "wisp_probe_h2d": [_P, _I, _I, ctypes.POINTER(ctypes.c_double)],
    "wisp_probe_h2d_engine": [_P, _I, _I, _I, ctypes.POINTER(ctypes.c_double)],
    "wisp_hbm_copy": [_P, _P, _U64, _P],
    "wisp_probe_hbm_read": [_U64, _I, ctypes.POINTER(ctypes.c_double)],
    "wisp_probe_mfma": [_I, ctypes.POINTER(ctypes.c_double)],
    "wisp_decode_fp8": [_P, _P, _I, _P],
    "wisp_debug_fail_slot_alloc": [_P, _I],
    "wisp_debug_poison_victims": [_P, _I],
    "wisp_route_topk_noalloc": [_P, _P, _I, _I, _I, _I, _I, _I, _I, _I, _P, _P, _P],
    "wisp_predictor_create": [_I, _I, _I, ctypes.c_double, ctypes.POINTER(_P)],
    "wisp_predictor_destroy": [_P],
    "wisp_predictor_shape": [_P, ctypes.POINTER(_I), ctypes.POINTER(_I)],
    "wisp_predictor_observe": [_P, _I, _P, _I],
    "wisp_predictor_end_pass": [_P],
    "wisp_predictor_predict": [_P, _I, _I, _P, ctypes.POINTER(_I), _P],
    "wisp_prefetch": [_P, _I, _P, _I],
    "wisp_set_prefetch": [_P, _I, _P, _I],
    "wisp_set_prefetch_hints": [_P, _P, _I],
    "wisp_prefetch_requests": [_P, _I, _P, _I, ctypes.POINTER(_I)],
    "wisp_prefetch_stats": [_P, ctypes.POINTER(_U64), ctypes.POINTER(_U64)],
    "wisp_last_error": [],
    "wisp_slot_table_create": [_I, _I],
    "wisp_slot_table_destroy": [_P],
    "wisp_slot_table_step": [_P, _P, _I, _P, _P, _P, _P, _P, _P],
    "wisp_slot_table_resize": [_P, _I],
    "wisp_slot_table_prefetch": [_P, _P, _I, _P, _P],
    "wisp_slot_table_slot_of": [_P, _I],
    "wisp_slot_table_expert_in": [_P, _I],
    "wisp_slot_table_tick": [_P, _I],
    "wisp_slot_table_cap": [_P],
}
_RESTYPES = {"wisp_last_error": ctypes.c_char_p, "wisp_slot_table_create": _P, "wisp_slot_table_destroy": None,
             "wisp_slot_table_tick": _U64}


def lib():
    """Load libwisp.so (raises if it is not built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build(); "
                               "there is no fallback path")
        L = ctypes.CDLL(LIB_PATH)
        for name, args in _SIGS.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = _RESTYPES.get(name, ctypes.c_int)
        _lib = L
    return _lib


def last_error():
    return lib().wisp_last_error().decode()


def check(status, func):
    if status != OK:
        raise WispError(status, func, last_error())


def _ptr(x):
    """Address of a torch tensor, numpy array, int or None."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if isinstance(x, np.ndarray):
        return x.ctypes.data
    return x.data_ptr()


def _stream(s):
    if s is None:
        return None
    return s.cuda_stream if hasattr(s, "cuda_stream") else int(s)


def desc_of(wl, max_tokens=None, pageable=False):
    return ModelDesc(wl.L, wl.d, wl.I, wl.N, wl.k, wl.n_groups, wl.topk_groups, int(wl.has_shared), wl.route,
                     wl.w_dtype, wl.x_dtype, max_tokens or wl.T, int(bool(pageable)))


def expert_bytes(desc):
    b = _U64()
    check(lib().wisp_expert_bytes(ctypes.byref(desc), ctypes.byref(b)), "wisp_expert_bytes")
    return b.value


class Context:
    """Owner of a wisp_ctx; method names follow the C ABI without the ``wisp_`` prefix."""

    def __init__(self, desc):
        self.desc = desc
        h = _P()
        check(lib().wisp_create(ctypes.byref(desc), ctypes.byref(h)), "wisp_create")
        self.h = h

    def close(self):
        if self.h:
            check(lib().wisp_destroy(self.h), "wisp_destroy")
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def expert_host_ptr(self, layer, expert):
        p = _P()
        b = _U64()
        check(lib().wisp_expert_host_ptr(self.h, layer, expert, ctypes.byref(p), ctypes.byref(b)),
              "wisp_expert_host_ptr")
        return p.value, b.value

    def masters_ready(self):
        check(lib().wisp_masters_ready(self.h), "wisp_masters_ready")

    def router_weights(self, layer, wr_dev):
        check(lib().wisp_router_weights(self.h, layer, _ptr(wr_dev)), "wisp_router_weights")

    def set_budget(self, expert_bytes):
        c = _I()
        check(lib().wisp_set_budget(self.h, int(expert_bytes), ctypes.byref(c)), "wisp_set_budget")
        return c.value

    def preload(self):
        check(lib().wisp_preload(self.h), "wisp_preload")

    def set_pager(self, pager):
        """PAGER_HOST (host slot table, hipMemcpyAsync fills) or PAGER_DEVICE (slot table in HBM)."""
        check(lib().wisp_set_pager(self.h, int(pager)), "wisp_set_pager")

    def set_fusion(self, on):
        """Down projection fused with the combine for single-token steps (default on), or separate kernels."""
        check(lib().wisp_set_fusion(self.h, int(bool(on))), "wisp_set_fusion")

    def route_topk(self, layer, x, T, idx, w, idx_host=None, stream=None):
        check(lib().wisp_route_topk(self.h, layer, _ptr(x), T, _ptr(idx), _ptr(w), _ptr(idx_host), _stream(stream)),
              "wisp_route_topk")

    def page_in(self, layer, ids_host, T):
        ids = np.ascontiguousarray(ids_host, dtype=np.int32)
        st = PageStats()
        check(lib().wisp_page_in(self.h, layer, ids.ctypes.data, T, ctypes.byref(st)), "wisp_page_in")
        return st.as_dict()

    def moe_forward(self, layer, x, T, w, y, stream=None):
        st = PageStats()
        check(lib().wisp_moe_forward(self.h, layer, _ptr(x), T, _ptr(w), _ptr(y), _stream(stream), ctypes.byref(st)),
              "wisp_moe_forward")
        return st.as_dict()

    def decode_step(self, x, T, idx, w, y, stream=None, stats=None):
        check(lib().wisp_decode_step(self.h, _ptr(x), T, _ptr(idx), _ptr(w), _ptr(y), _stream(stream), _ptr(stats)),
              "wisp_decode_step")

    def offload_begin(self, expert_bytes, mode=0):
        """Static offload at this VRAM expert budget (mode OFFLOAD_BULK or OFFLOAD_ZERO_COPY); returns
        the number of resident layers."""
        r = _I()
        check(lib().wisp_offload_begin(self.h, int(expert_bytes), int(mode), ctypes.byref(r)), "wisp_offload_begin")
        return r.value

    def offload_step(self, x, T, idx, w, y, stream=None):
        check(lib().wisp_offload_step(self.h, _ptr(x), T, _ptr(idx), _ptr(w), _ptr(y), _stream(stream)),
              "wisp_offload_step")

    def offload_end(self):
        check(lib().wisp_offload_end(self.h), "wisp_offload_end")

    def stats(self, layer):
        st = PageStats()
        check(lib().wisp_get_stats(self.h, layer, ctypes.byref(st)), "wisp_get_stats")
        return st.as_dict()

    def reset_stats(self):
        check(lib().wisp_reset_stats(self.h), "wisp_reset_stats")

    def cap(self):
        c = _I()
        check(lib().wisp_get_cap(self.h, ctypes.byref(c)), "wisp_get_cap")
        return c.value

    def slot_of(self, layer, expert):
        s = _I()
        check(lib().wisp_slot_of(self.h, layer, expert, ctypes.byref(s)), "wisp_slot_of")
        return s.value

    def expert_in_slot(self, layer, slot):
        e = _I()
        check(lib().wisp_expert_in_slot(self.h, layer, slot, ctypes.byref(e)), "wisp_expert_in_slot")
        return e.value

    def read_slot(self, layer, slot, nbytes):
        out = np.empty(nbytes, np.uint8)
        check(lib().wisp_read_slot(self.h, layer, slot, out.ctypes.data), "wisp_read_slot")
        return out

    def set_profiling(self, class_mask):
        """class_mask: bit c times kernel class c (1 << K_FFN_GATEUP, ...); True = every class; 0 = off."""
        mask = (1 << len(KERNEL_CLASS_NAMES)) - 1 if class_mask is True else int(class_mask)
        check(lib().wisp_set_profiling(self.h, mask), "wisp_set_profiling")

    def kernel_times(self, kclass):
        ms = ctypes.c_double()
        n = _U64()
        b = _U64()
        f = _U64()
        check(lib().wisp_kernel_times(self.h, kclass, ctypes.byref(ms), ctypes.byref(n), ctypes.byref(b),
                                      ctypes.byref(f)), "wisp_kernel_times")
        return dict(total_ms=ms.value, launches=n.value, bytes=b.value, flops=f.value)

    def reset_kernel_times(self):
        check(lib().wisp_reset_kernel_times(self.h), "wisp_reset_kernel_times")

    def probe_h2d(self, count, reps, engine=None):
        """Median host->device GB/s over `reps` rounds of `count` expert blobs: the copy engine (default,
        wisp_probe_h2d) or engine=LINK_CUS (compute-unit streaming, as the token-batch fills)."""
        g = ctypes.c_double()
        if engine is None:
            check(lib().wisp_probe_h2d(self.h, count, reps, ctypes.byref(g)), "wisp_probe_h2d")
        else:
            check(lib().wisp_probe_h2d_engine(self.h, count, reps, engine, ctypes.byref(g)), "wisp_probe_h2d_engine")
        return g.value

    def debug_poison_victims(self, on):
        """Overwrite every victim slot with NaN bytes after its write-after-read wait, before its fill."""
        check(lib().wisp_debug_poison_victims(self.h, int(bool(on))), "wisp_debug_poison_victims")

    def debug_fail_slot_alloc(self, n):
        check(lib().wisp_debug_fail_slot_alloc(self.h, n), "wisp_debug_fail_slot_alloc")

    def prefetch(self, layer, ids):
        ids = np.ascontiguousarray(np.asarray(ids, dtype=np.int32).ravel())
        check(lib().wisp_prefetch(self.h, layer, ids.ctypes.data if ids.size else None, ids.size), "wisp_prefetch")

    def set_prefetch(self, mode, predictor=None, depth=0):
        """PREFETCH_OFF, PREFETCH_PREDICTOR (with a Predictor and a depth) or PREFETCH_HINTS."""
        check(lib().wisp_set_prefetch(self.h, int(mode), predictor.h if predictor is not None else None, int(depth)),
              "wisp_set_prefetch")

    def set_prefetch_hints(self, ids):
        """ids [L, n] (-1 = none): the experts prefetched per layer during the next decode step."""
        ids = np.ascontiguousarray(np.asarray(ids, dtype=np.int32))
        n = ids.shape[1] if ids.ndim == 2 else 0
        check(lib().wisp_set_prefetch_hints(self.h, ids.ctypes.data if ids.size else None, n),
              "wisp_set_prefetch_hints")

    def prefetch_requests(self, layer):
        """The ids the last decode step asked to prefetch for `layer`."""
        out = np.zeros(max(self.desc.n_experts, 1), np.int32)
        n = _I()
        check(lib().wisp_prefetch_requests(self.h, int(layer), out.ctypes.data, out.size, ctypes.byref(n)),
              "wisp_prefetch_requests")
        return out[:n.value].copy()

    def prefetch_stats(self):
        a, b = _U64(), _U64()
        check(lib().wisp_prefetch_stats(self.h, ctypes.byref(a), ctypes.byref(b)), "wisp_prefetch_stats")
        return dict(issued=a.value, useful=b.value)


class Predictor:
    """The co-activation predictor (wisp_predictor_*): host code, no GPU."""

    def __init__(self, n_layers, n_experts, horizon, gamma):
        self.h = _P()
        check(lib().wisp_predictor_create(int(n_layers), int(n_experts), int(horizon), float(gamma),
                                          ctypes.byref(self.h)), "wisp_predictor_create")

    def close(self):
        if self.h:
            check(lib().wisp_predictor_destroy(self.h), "wisp_predictor_destroy")
            self.h = _P()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def observe(self, layer, ids):
        ids = np.ascontiguousarray(np.asarray(ids, dtype=np.int32).ravel())
        check(lib().wisp_predictor_observe(self.h, int(layer), ids.ctypes.data if ids.size else None, ids.size),
              "wisp_predictor_observe")

    def end_pass(self):
        check(lib().wisp_predictor_end_pass(self.h), "wisp_predictor_end_pass")

    def predict(self, layer, depth):
        """(ids, scores) of the `depth` best-scoring experts of `layer` (score desc, id asc; positive only)."""
        ids = np.zeros(max(depth, 1), np.int32)
        sc = np.zeros(max(depth, 1), np.float64)
        n = _I()
        check(lib().wisp_predictor_predict(self.h, int(layer), int(depth), ids.ctypes.data, ctypes.byref(n),
                                           sc.ctypes.data), "wisp_predictor_predict")
        return ids[:n.value].copy(), sc[:n.value].copy()


def probe_hbm_read(nbytes, launches):
    """Mean microseconds per launch of a plain streaming read of nbytes (a multiple of 16), launched
    back to back over windows of a buffer beyond the last-level cache (wisp_probe_hbm_read)."""
    us = ctypes.c_double()
    check(lib().wisp_probe_hbm_read(int(nbytes), int(launches), ctypes.byref(us)), "wisp_probe_hbm_read")
    return us.value


def probe_mfma(launches):
    """Dense bf16 matrix-core TFLOP/s the device sustains on register operands (wisp_probe_mfma)."""
    tf = ctypes.c_double()
    check(lib().wisp_probe_mfma(int(launches), ctypes.byref(tf)), "wisp_probe_mfma")
    return tf.value


def hbm_copy(src, dst, nbytes, stream=None):
    check(lib().wisp_hbm_copy(_ptr(src), _ptr(dst), int(nbytes), _stream(stream)), "wisp_hbm_copy")


NOALLOC_MAX_LOGITS = 524288


def route_topk_noalloc(wr, x, x_dtype, T, N, d, k, route, n_groups, topk_groups, idx, w, stream=None):
    """Route T tokens without a context and without allocating (wisp_route_topk_noalloc): the
    kernels' scratch is the library's fixed device array, shared by every call on the device."""
    check(lib().wisp_route_topk_noalloc(_ptr(wr), _ptr(x), int(x_dtype), int(T), int(N), int(d), int(k), int(route),
                                        int(n_groups), int(topk_groups), _ptr(idx), _ptr(w), _stream(stream)),
          "wisp_route_topk_noalloc")


def decode_fp8(codes_dev, out_dev, n, stream=None):
    check(lib().wisp_decode_fp8(_ptr(codes_dev), _ptr(out_dev), n, _stream(stream)), "wisp_decode_fp8")


class SlotTable:
    """The pager's host slot table through its C export (pure host code, no GPU)."""

    def __init__(self, N, C):
        self.N = N
        self.h = lib().wisp_slot_table_create(N, C)
        if not self.h:
            raise ValueError(f"invalid slot table N={N} C={C}")

    def __del__(self):
        if getattr(self, "h", None):
            lib().wisp_slot_table_destroy(self.h)
            self.h = None

    def step(self, ids):
        ids = np.ascontiguousarray(np.asarray(ids, np.int32).ravel())
        n = ids.size
        h, m, c = _I(), _I(), _I()
        mi = np.zeros(max(n, 1), np.int32)
        ms = np.zeros(max(n, 1), np.int32)
        mc = np.zeros(max(n, 1), np.int32)
        rc = lib().wisp_slot_table_step(self.h, ids.ctypes.data, n, ctypes.byref(h), ctypes.byref(m), ctypes.byref(c),
                                        mi.ctypes.data, ms.ctypes.data, mc.ctypes.data)
        if rc != 0:
            raise ValueError("bad expert id")
        k = m.value
        return dict(hits=h.value, misses=k, chunks=c.value, miss_ids=mi[:k].copy(), miss_slots=ms[:k].copy(),
                    miss_chunk=mc[:k].copy())

    def prefetch(self, ids):
        """Speculative page-in; returns (fill_ids, fill_slots) in copy order."""
        ids = np.ascontiguousarray(np.asarray(ids, np.int32).ravel())
        fi = np.zeros(max(ids.size, 1), np.int32)
        fs = np.zeros(max(ids.size, 1), np.int32)
        m = lib().wisp_slot_table_prefetch(self.h, ids.ctypes.data if ids.size else None, ids.size, fi.ctypes.data,
                                           fs.ctypes.data)
        if m < 0:
            raise ValueError("bad expert id")
        return fi[:m].copy(), fs[:m].copy()

    def resize(self, C):
        if lib().wisp_slot_table_resize(self.h, C) != 0:
            raise ValueError(f"invalid cap {C}")

    def slot_of(self, e):
        return lib().wisp_slot_table_slot_of(self.h, e)

    def expert_in(self, s):
        return lib().wisp_slot_table_expert_in(self.h, s)

    def tick(self, s):
        return int(lib().wisp_slot_table_tick(self.h, s))

    @property
    def cap(self):
        return lib().wisp_slot_table_cap(self.h)


# ------------------------------------------------------------------------------------------------
# Expert <-> KV allocator (wisp_mvwsa.h)
# ------------------------------------------------------------------------------------------------
def miss_curve(ids, n_experts, upper=False):
    """Expert miss curve m(C), C = 0..n_experts, of one layer's routing trace ids [steps, refs]; with
    upper=True also the upper-bound curve: (lower, upper)."""
    ids = np.ascontiguousarray(np.asarray(ids, dtype=np.int32))
    if ids.ndim == 1:
        ids = ids[:, None]
    out = np.zeros(n_experts + 1, np.uint64)
    up = np.zeros(n_experts + 1, np.uint64) if upper else None
    check(lib().wisp_miss_curve(ids.ctypes.data, ids.shape[0], ids.shape[1], n_experts, out.ctypes.data,
                                up.ctypes.data if upper else None), "wisp_miss_curve")
    return (out, up) if upper else out


def mvwsa_configure(B, a, b, kv_min, c_exp, c_kv, m_exp, m_kv):
    """MV-WSA startup configurator (Eqs. 3-5); returns dict(cap, kv_blocks, kv_bytes, f, latency, floor_binding)."""
    m_exp = np.ascontiguousarray(np.asarray(m_exp, dtype=np.uint64))
    m_kv = np.ascontiguousarray(np.asarray(m_kv, dtype=np.float64))
    pr = MvwsaProblem(int(B), int(a), int(b), int(kv_min), float(c_exp), float(c_kv), m_exp.size - 1, m_kv.size)
    out = MvwsaSplit()
    check(lib().wisp_mvwsa_configure(ctypes.byref(pr), m_exp.ctypes.data, m_kv.ctypes.data, ctypes.byref(out)),
          "wisp_mvwsa_configure")
    return dict(cap=out.cap, kv_blocks=out.kv_blocks, kv_bytes=out.kv_bytes, f=out.f, latency=out.latency,
                floor_binding=bool(out.floor_binding))


def resize_target(B, a, b, kv_min, headroom, cap_min, cap_max, dead_zone, peak_blocks, cap_now):
    """Dual-resize control law (App. B, Eqs. 6-8); returns (cap, kv_blocks, move)."""
    law = ResizeLaw(int(B), int(a), int(b), int(kv_min), float(headroom), int(cap_min), int(cap_max), int(dead_zone))
    c, k, m = _I(), ctypes.c_int64(), _I()
    check(lib().wisp_resize_target(ctypes.byref(law), int(peak_blocks), int(cap_now), ctypes.byref(c), ctypes.byref(k),
                                   ctypes.byref(m)), "wisp_resize_target")
    return c.value, k.value, bool(m.value)


class KvPool:
    """A KV block pool in device memory (wisp_kv_pool_*); the KV side of the budget."""

    def __init__(self, block_bytes, blocks):
        self.h = _P()
        check(lib().wisp_kv_pool_create(int(block_bytes), int(blocks), ctypes.byref(self.h)), "wisp_kv_pool_create")
        self.block_bytes = int(block_bytes)

    @property
    def blocks(self):
        n = ctypes.c_int64()
        check(lib().wisp_kv_pool_blocks(self.h, ctypes.byref(n)), "wisp_kv_pool_blocks")
        return n.value

    def resize(self, blocks):
        check(lib().wisp_kv_pool_resize(self.h, int(blocks)), "wisp_kv_pool_resize")

    def close(self):
        if self.h:
            check(lib().wisp_kv_pool_destroy(self.h), "wisp_kv_pool_destroy")
            self.h = _P()


def dual_resize(ctx, pool, cap_new, kv_blocks_new):
    """The drained-barrier move of App. B between the expert scratch of ctx and the KV pool."""
    check(lib().wisp_dual_resize(ctx.h, pool.h, int(cap_new), int(kv_blocks_new)), "wisp_dual_resize")


class Controller:
    """The online dual-resize controller (wisp_controller_*): observe the KV blocks in use after each
    decode step; barrier() at a drained barrier applies the control law to ctx and pool (or only
    decides when both are None)."""

    def __init__(self, B, a, b, kv_min, headroom, cap_min, cap_max, dead_zone, cap_now, kv_now):
        law = ResizeLaw(int(B), int(a), int(b), int(kv_min), float(headroom), int(cap_min), int(cap_max),
                        int(dead_zone))
        self.h = _P()
        check(lib().wisp_controller_create(ctypes.byref(law), int(cap_now), int(kv_now), ctypes.byref(self.h)),
              "wisp_controller_create")

    def observe(self, kv_blocks_in_use):
        check(lib().wisp_controller_observe(self.h, int(kv_blocks_in_use)), "wisp_controller_observe")

    def barrier(self, ctx=None, pool=None):
        """Returns (cap, kv_blocks, moved, peak): the split after the barrier, 1 moved / 0 none / -1 a
        failed move skipped, and the peak the law used (-1: nothing observed)."""
        c, k, m, p = _I(), ctypes.c_int64(), _I(), ctypes.c_int64()
        check(lib().wisp_controller_barrier(self.h, ctx.h if ctx is not None else None,
                                            pool.h if pool is not None else None, ctypes.byref(c), ctypes.byref(k),
                                            ctypes.byref(m), ctypes.byref(p)), "wisp_controller_barrier")
        return c.value, k.value, m.value, p.value

    def close(self):
        if self.h:
            check(lib().wisp_controller_destroy(self.h), "wisp_controller_destroy")
            self.h = _P()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


# ------------------------------------------------------------------------------------------------
# Harness: one workload end to end
# ------------------------------------------------------------------------------------------------
class DecodeRun:
    """Context + inputs for one workload on one GPU.

    generate() fills the pinned masters with the seeded generator (in parallel, straight into the
    library's pinned memory), uploads router weights and the hidden states of every step
    ([steps, L, T, d] on the device), and declares the masters ready.
    """

    def __init__(self, wl, device=0, max_tokens=None, steps=None, pageable=False):
        import torch
        self.torch = torch
        self.wl = wl
        self.device = device
        torch.cuda.set_device(device)
        self.dev = torch.device("cuda", device)
        self.stream = torch.cuda.Stream(device=self.dev)
        self.steps = steps or wl.steps
        self.pageable = bool(pageable)
        self.ctx = Context(desc_of(wl, max_tokens, pageable))
        self.blob_bytes = expert_bytes(self.ctx.desc)
        self.gen_seconds = None

    def close(self):
        if self.ctx is not None:
            self.ctx.close()
            self.ctx = None

    def master_ptrs(self, layer):
        return [self.ctx.expert_host_ptr(layer, e)[0] for e in range(self.wl.N)]

    def shared_ptr(self, layer):
        return self.ctx.expert_host_ptr(layer, -1)[0] if self.wl.has_shared else None

    def master_blob(self, layer, expert):
        """Copy of a master blob as a numpy uint8 array."""
        p, n = self.ctx.expert_host_ptr(layer, expert)
        return np.ctypeslib.as_array((ctypes.c_uint8 * n).from_address(p)).copy()

    def generate(self, threads=0, inputs=True):
        from . import datagen as dg
        torch = self.torch
        wl = self.wl
        t0 = time.time()
        layers, experts, ptrs = [], [], []
        for l in range(wl.L):
            for e in range(wl.N):
                layers.append(l)
                experts.append(e)
                ptrs.append(self.ctx.expert_host_ptr(l, e)[0])
            if wl.has_shared:
                layers.append(l)
                experts.append(dg.SHARED_EXPERT)
                ptrs.append(self.ctx.expert_host_ptr(l, -1)[0])
        dg.fill_blobs(wl.seed, layers, experts, ptrs, wl.w_dtype, wl.d, wl.I, threads=threads)
        self.ctx.masters_ready()
        self.wr_host = np.stack([dg.router_weights(wl.seed, l, wl.N, wl.d) for l in range(wl.L)])
        self.wr_dev = torch.from_numpy(self.wr_host).to(self.dev)
        for l in range(wl.L):
            self.ctx.router_weights(l, self.wr_dev[l])
        if inputs:
            if wl.prefill:
                x = dg.prefill_inputs(wl.seed, wl.L, wl.T, wl.d, wl.x_dtype, threads=threads)
                self.x_host = x[:, None]                      # [L, 1, T, d]
            else:
                self.x_host = dg.decode_inputs(wl.seed, wl.L, self.steps, wl.T, wl.d, wl.x_dtype, threads=threads)
            xs = np.ascontiguousarray(self.x_host.transpose(1, 0, 2, 3))  # [S, L, T, d]
            xt = torch.from_numpy(xs.view(np.int16) if xs.dtype == np.uint16 else xs)
            self.x_dev = xt.to(self.dev)
        torch.cuda.synchronize(self.dev)
        self.gen_seconds = time.time() - t0

    def set_cap(self, cap):
        return self.ctx.set_budget(cap * self.wl.L * self.blob_bytes)

    def decode(self, record=True, steps=None, start=0, stats=True, hints=None, prefetch_log=False):
        """Run decode steps [start, start + steps) through wisp_decode_step.

        Returns numpy arrays idx [S, L, T, k], w [S, L, T, k], y [S, L, T, d] (if record), and per
        (step, layer) hits/misses.  hints [S, L, n]: prefetch hints set before each step (prefetch
        mode PREFETCH_HINTS); prefetch_log: also return the ids each step asked to prefetch per layer
        (``requests[s][l]``)."""
        torch = self.torch
        wl = self.wl
        S = steps if steps is not None else self.steps - start
        T, L, k, d = wl.T, wl.L, wl.k, wl.d
        nrec = S if record else 1
        idx = torch.zeros((nrec, L, T, k), dtype=torch.int32, device=self.dev)
        w = torch.zeros((nrec, L, T, k), dtype=torch.float32, device=self.dev)
        y = torch.zeros((nrec, L, T, d), dtype=torch.float32, device=self.dev)
        st = (PageStats * L)()
        hits = np.zeros((S, L), np.int64)
        misses = np.zeros((S, L), np.int64)
        chunks = np.zeros((S, L), np.int64)
        requests = []
        torch.cuda.synchronize(self.dev)
        with torch.cuda.stream(self.stream):
            for s in range(S):
                r = s if record else 0
                if hints is not None:
                    self.ctx.set_prefetch_hints(hints[s])
                self.ctx.decode_step(self.x_dev[start + s], T, idx[r], w[r], y[r], self.stream,
                                     ctypes.addressof(st) if stats else None)
                if stats:
                    for l in range(L):
                        hits[s, l] = st[l].hits
                        misses[s, l] = st[l].misses
                        chunks[s, l] = st[l].chunks
                if prefetch_log:
                    requests.append([self.ctx.prefetch_requests(l) for l in range(L)])
        self.stream.synchronize()
        out = dict(hits=hits, misses=misses, chunks=chunks)
        if prefetch_log:
            out["requests"] = requests
        if record:
            out.update(idx=idx.cpu().numpy(), w=w.cpu().numpy(), y=y.cpu().numpy())
        return out

    def offload(self, record=True, steps=None, start=0):
        """Run decode steps [start, start + steps) through the static-offload arm (wisp_offload_begin
        must have been called).  Returns idx, w, y as decode() does (if record)."""
        torch = self.torch
        wl = self.wl
        S = steps if steps is not None else self.steps - start
        T, L, k, d = wl.T, wl.L, wl.k, wl.d
        nrec = S if record else 1
        idx = torch.zeros((nrec, L, T, k), dtype=torch.int32, device=self.dev)
        w = torch.zeros((nrec, L, T, k), dtype=torch.float32, device=self.dev)
        y = torch.zeros((nrec, L, T, d), dtype=torch.float32, device=self.dev)
        torch.cuda.synchronize(self.dev)
        with torch.cuda.stream(self.stream):
            for s in range(S):
                r = s if record else 0
                self.ctx.offload_step(self.x_dev[start + s], T, idx[r], w[r], y[r], self.stream)
        self.stream.synchronize()
        out = {}
        if record:
            out.update(idx=idx.cpu().numpy(), w=w.cpu().numpy(), y=y.cpu().numpy())
        return out
