"""ORACLE — test infrastructure, not part of the product.

ctypes binding of ``liboracle.so`` (built from ``oracle.c``): a plain fp64 CPU reference of the
paged MoE layer (fully resident router + expert FFN + combine) and an LRU simulator that runs
Algorithm 1 of WiSP (arXiv 2606.21868, Sec. 3.2).  Only ``tests/``, ``__graft_entry__.smoke()``
and the CPU-baseline leg of ``bench.py`` may import this package.  It never imports the HIP
path, and the HIP path never imports it.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

ROUTE_SOFTMAX_RENORM, ROUTE_TOPK_SOFTMAX, ROUTE_SIGMOID_GROUP = 0, 1, 2
F32, BF16, FP8 = 0, 1, 2

_p = ctypes.c_void_p
_i = ctypes.c_int


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError(f"{_LIB_PATH} is not built; run __graft_entry__.build()")
        L = ctypes.CDLL(_LIB_PATH)
        L.oracle_bf16_value.argtypes = [ctypes.c_uint16]
        L.oracle_bf16_value.restype = ctypes.c_double
        L.oracle_e4m3_value.argtypes = [ctypes.c_uint8]
        L.oracle_e4m3_value.restype = ctypes.c_double
        L.oracle_route.argtypes = [_i, _i, _i, _i, _i, _i, _p, _i, _p, _p, _p, _p, _p, _p]
        L.oracle_expert.argtypes = [_p, _i, _i, _i, _i, _p, _p, _p]
        L.oracle_moe_layer.argtypes = [_i, _i, _i, _i, _i, _i, _i, _i, _p, _p, _p, _i, _p, _i, _p, _p, _p,
                                       _p, _p]
        L.oracle_moe_layer_routed.argtypes = [_i, _i, _i, _i, _i, _i, _p, _p, _p, _i, _p, _i, _p, _p, _p]
        L.oracle_route_gates.argtypes = [_i, _i, _i, _p, _i, _p, _i, _p, _p]
        L.oracle_lru_new.argtypes = [_i, _i]
        L.oracle_lru_new.restype = _p
        L.oracle_lru_free.argtypes = [_p]
        L.oracle_lru_slot.argtypes = [_p, _i]
        L.oracle_lru_expert_in.argtypes = [_p, _i]
        L.oracle_lru_tick.argtypes = [_p, _i]
        L.oracle_lru_tick.restype = ctypes.c_uint64
        L.oracle_lru_clock.argtypes = [_p]
        L.oracle_lru_clock.restype = ctypes.c_uint64
        L.oracle_lru_cap.argtypes = [_p]
        L.oracle_lru_step.argtypes = [_p, _p, _i, _p, _p, _p, _p, _p]
        L.oracle_lru_resize.argtypes = [_p, _i]
        L.oracle_lru_prefetch.argtypes = [_p, _p, _i, _p, _p]
        L.oracle_num_threads.argtypes = []
        _lib = L
    return _lib


def _ptr(a):
    return a.ctypes.data if isinstance(a, np.ndarray) else int(a)


def bf16_value(bits):
    return lib().oracle_bf16_value(int(bits))


def e4m3_value(code):
    return lib().oracle_e4m3_value(int(code))


def x_dtype_of(x):
    return F32 if x.dtype == np.float32 else BF16


def route(variant, Wr, x, k, n_groups=1, topk_groups=1):
    """Route one token.  Returns (idx[k], gates[k], scores[N], margin, group_margin)."""
    Wr = np.ascontiguousarray(Wr, dtype=np.float32)
    x = np.ascontiguousarray(x)
    N, d = Wr.shape
    idx = np.zeros(k, np.int32)
    g = np.zeros(k, np.float64)
    sc = np.zeros(N, np.float64)
    m = np.zeros(1, np.float64)
    gm = np.zeros(1, np.float64)
    lib().oracle_route(variant, N, d, k, n_groups, topk_groups, Wr.ctypes.data, x_dtype_of(x), x.ctypes.data,
                       idx.ctypes.data, g.ctypes.data, sc.ctypes.data, m.ctypes.data, gm.ctypes.data)
    return idx, g, sc, float(m[0]), float(gm[0])


def expert(blob, w_dtype, d, I, x, return_h=False):
    """o = W2 (silu(W1 x) * W3 x) for one token, fp64.  blob: uint8 array or host address."""
    x = np.ascontiguousarray(x)
    o = np.zeros(d, np.float64)
    h = np.zeros(I, np.float64)
    lib().oracle_expert(_ptr(blob), w_dtype, d, I, x_dtype_of(x), x.ctypes.data, o.ctypes.data, h.ctypes.data)
    return (o, h) if return_h else o


def moe_layer(variant, blobs, Wr, x, k, I, w_dtype, shared_blob=None, n_groups=1, topk_groups=1):
    """Fully resident layer for x [T, d].  blobs: list of N blob arrays or host addresses.
    Returns (idx [T,k], gates [T,k], y [T,d] fp64, margins [T], group_margins [T])."""
    Wr = np.ascontiguousarray(Wr, dtype=np.float32)
    x = np.ascontiguousarray(x)
    N, d = Wr.shape
    T = x.shape[0]
    arr = (ctypes.c_void_p * N)(*[_ptr(b) for b in blobs])
    idx = np.zeros((T, k), np.int32)
    g = np.zeros((T, k), np.float64)
    y = np.zeros((T, d), np.float64)
    mg = np.zeros(T, np.float64)
    gmg = np.zeros(T, np.float64)
    sh = _ptr(shared_blob) if shared_blob is not None else None
    lib().oracle_moe_layer(variant, N, d, I, k, n_groups, topk_groups, w_dtype, arr, sh, Wr.ctypes.data,
                           x_dtype_of(x), x.ctypes.data, T, idx.ctypes.data, g.ctypes.data, y.ctypes.data,
                           mg.ctypes.data, gmg.ctypes.data)
    return idx, g, y, mg, gmg


def route_gates(variant, Wr, x, idx):
    """Gates of a given routed set idx[k] (rank order) of one token, by the variant's rule."""
    Wr = np.ascontiguousarray(Wr, dtype=np.float32)
    x = np.ascontiguousarray(x)
    idx = np.ascontiguousarray(np.asarray(idx, dtype=np.int32).ravel())
    N, d = Wr.shape
    if idx.min(initial=0) < 0 or idx.max(initial=0) >= N:
        raise ValueError("expert id out of range")
    g = np.zeros(idx.size, np.float64)
    lib().oracle_route_gates(variant, N, d, Wr.ctypes.data, x_dtype_of(x), x.ctypes.data, idx.size,
                             idx.ctypes.data, g.ctypes.data)
    return g


def moe_layer_routed(variant, blobs, Wr, x, idx, I, w_dtype, shared_blob=None):
    """The fully resident layer evaluated on a given routing idx [T, k] (rank order) instead of the
    oracle's own selection: gates by the variant's rule over that set, combine in that order.
    Returns (gates [T,k], y [T,d] fp64)."""
    Wr = np.ascontiguousarray(Wr, dtype=np.float32)
    x = np.ascontiguousarray(x)
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    N, d = Wr.shape
    T, k = idx.shape
    if x.shape[0] != T or idx.min(initial=0) < 0 or idx.max(initial=0) >= N:
        raise ValueError("routing does not match the tokens or the expert count")
    arr = (ctypes.c_void_p * N)(*[_ptr(b) for b in blobs])
    g = np.zeros((T, k), np.float64)
    y = np.zeros((T, d), np.float64)
    sh = _ptr(shared_blob) if shared_blob is not None else None
    lib().oracle_moe_layer_routed(variant, N, d, I, k, w_dtype, arr, sh, Wr.ctypes.data, x_dtype_of(x),
                                  x.ctypes.data, T, idx.ctypes.data, g.ctypes.data, y.ctypes.data)
    return g, y


class LRU:
    """Algorithm 1 simulator for one layer (cold start)."""

    def __init__(self, N, C):
        self.N = N
        self._h = lib().oracle_lru_new(N, C)
        if not self._h:
            raise ValueError(f"invalid LRU shape N={N} C={C}")

    def __del__(self):
        if getattr(self, "_h", None):
            lib().oracle_lru_free(self._h)
            self._h = None

    @property
    def cap(self):
        return lib().oracle_lru_cap(self._h)

    def step(self, ids):
        """Returns dict(hits, misses, chunks, miss_ids, miss_slots) for one layer-step."""
        ids = np.ascontiguousarray(np.asarray(ids, dtype=np.int32).ravel())
        n = ids.size
        h = np.zeros(1, np.int32)
        m = np.zeros(1, np.int32)
        c = np.zeros(1, np.int32)
        mi = np.zeros(max(n, 1), np.int32)
        ms = np.zeros(max(n, 1), np.int32)
        rc = lib().oracle_lru_step(self._h, ids.ctypes.data, n, h.ctypes.data, m.ctypes.data, c.ctypes.data,
                                   mi.ctypes.data, ms.ctypes.data)
        if rc != 0:
            raise ValueError("expert id out of range")
        nm = int(m[0])
        return dict(hits=int(h[0]), misses=nm, chunks=int(c[0]), miss_ids=mi[:nm].copy(),
                    miss_slots=ms[:nm].copy())

    def prefetch(self, ids):
        """Speculative prefetch; returns (fill_ids, fill_slots) in copy order."""
        ids = np.ascontiguousarray(np.asarray(ids, dtype=np.int32).ravel())
        fi = np.zeros(max(ids.size, 1), np.int32)
        fs = np.zeros(max(ids.size, 1), np.int32)
        m = lib().oracle_lru_prefetch(self._h, ids.ctypes.data, ids.size, fi.ctypes.data, fs.ctypes.data)
        if m < 0:
            raise ValueError("expert id out of range")
        return fi[:m].copy(), fs[:m].copy()

    def slot(self, e):
        return lib().oracle_lru_slot(self._h, e)

    def resident(self):
        return {e for e in range(self.N) if self.slot(e) >= 0}

    def tick(self, slot):
        return int(lib().oracle_lru_tick(self._h, slot))

    def resize(self, C):
        if lib().oracle_lru_resize(self._h, C) != 0:
            raise ValueError(f"invalid cap {C}")


def num_threads():
    return lib().oracle_num_threads()
