"""Seeded synthetic inputs (ctypes binding of ``libwisp_datagen.so``).

Produces only input bytes (weights, router weights, hidden states); none of the MoE method's
arithmetic lives here.  The HIP path and the CPU oracle both read what it writes.
See ``datagen.c`` for the generator (Philox4x32-10 + Box-Muller) and the blob format.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libwisp_datagen.so")
_lib = None

# dtype codes shared by the blob format
F32, BF16, FP8 = 0, 1, 2
KIND_W1, KIND_W3, KIND_W2, KIND_WR, KIND_XAR, KIND_XIID = 1, 2, 3, 4, 5, 6
SHARED_EXPERT = 4095
WEIGHT_STD = 0.02
AR_RHO = 0.9

_c_u32 = ctypes.c_uint32
_c_u64 = ctypes.c_uint64
_c_int = ctypes.c_int
_c_p = ctypes.c_void_p


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError(f"{_LIB_PATH} is not built; run __graft_entry__.build()")
        L = ctypes.CDLL(_LIB_PATH)
        L.wdg_philox4x32_10.argtypes = [_c_p, _c_p, _c_p]
        L.wdg_normals.argtypes = [_c_u32, _c_int, _c_int, _c_int, _c_u64, _c_u64, _c_p]
        L.wdg_f32_to_bf16.argtypes = [ctypes.c_float]
        L.wdg_f32_to_bf16.restype = ctypes.c_uint16
        L.wdg_f32_to_e4m3.argtypes = [ctypes.c_float]
        L.wdg_f32_to_e4m3.restype = ctypes.c_uint8
        L.wdg_f32_to_bf16_array.argtypes = [_c_p, _c_p, _c_u64]
        L.wdg_f32_to_e4m3_array.argtypes = [_c_p, _c_p, _c_u64]
        L.wdg_blob_bytes.argtypes = [_c_int, _c_int, _c_int]
        L.wdg_blob_bytes.restype = _c_u64
        L.wdg_expert_blob.argtypes = [_c_u32, _c_int, _c_int, _c_int, _c_int, _c_int, ctypes.c_float, _c_p]
        L.wdg_expert_blobs.argtypes = [_c_u32, _c_int, _c_p, _c_p, _c_p, _c_int, _c_int, _c_int,
                                       ctypes.c_float, _c_int]
        L.wdg_router.argtypes = [_c_u32, _c_int, _c_int, _c_int, _c_p]
        L.wdg_decode_inputs.argtypes = [_c_u32, _c_int, _c_int, _c_int, _c_int, ctypes.c_double, _c_int, _c_p, _c_int]
        L.wdg_prefill_inputs.argtypes = [_c_u32, _c_int, _c_int, _c_int, _c_int, _c_p, _c_int]
        _lib = L
    return _lib


def philox4x32_10(ctr, key):
    c = np.asarray(ctr, dtype=np.uint32).copy()
    k = np.asarray(key, dtype=np.uint32).copy()
    o = np.zeros(4, dtype=np.uint32)
    lib().wdg_philox4x32_10(c.ctypes.data, k.ctypes.data, o.ctypes.data)
    return o


def normals(seed, kind, layer, expert, start, n):
    out = np.empty(n, dtype=np.float32)
    lib().wdg_normals(seed, kind, layer, expert, start, n, out.ctypes.data)
    return out


def f32_to_bf16(x):
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty(x.shape, dtype=np.uint16)
    lib().wdg_f32_to_bf16_array(x.ctypes.data, out.ctypes.data, x.size)
    return out


def f32_to_e4m3(x):
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty(x.shape, dtype=np.uint8)
    lib().wdg_f32_to_e4m3_array(x.ctypes.data, out.ctypes.data, x.size)
    return out


def blob_bytes(dtype, d, I):
    return int(lib().wdg_blob_bytes(dtype, d, I))


def expert_blob(seed, layer, expert, dtype, d, I, std=WEIGHT_STD):
    """One expert blob as a uint8 numpy array (W1 | W3 | W2 [| scales])."""
    out = np.empty(blob_bytes(dtype, d, I), dtype=np.uint8)
    lib().wdg_expert_blob(seed, layer, expert, dtype, d, I, std, out.ctypes.data)
    return out


def fill_blobs(seed, layers, experts, ptrs, dtype, d, I, std=WEIGHT_STD, threads=0):
    """Generate blobs straight into caller memory (e.g. pinned host masters)."""
    n = len(ptrs)
    la = np.asarray(layers, dtype=np.int32)
    ea = np.asarray(experts, dtype=np.int32)
    pa = (ctypes.c_void_p * n)(*[int(p) for p in ptrs])
    lib().wdg_expert_blobs(seed, n, la.ctypes.data, ea.ctypes.data, pa, dtype, d, I, std, threads)


def router_weights(seed, layer, N, d):
    out = np.empty((N, d), dtype=np.float32)
    lib().wdg_router(seed, layer, N, d, out.ctypes.data)
    return out


def decode_inputs(seed, L, S, T, d, dtype, rho=AR_RHO, threads=0):
    """AR(1) hidden states [L, S, T, d]: fp32 (dtype F32) or bf16 bits as uint16 (dtype BF16)."""
    np_dt = np.float32 if dtype == F32 else np.uint16
    out = np.empty((L, S, T, d), dtype=np_dt)
    lib().wdg_decode_inputs(seed, L, S, T, d, rho, dtype, out.ctypes.data, threads)
    return out


def prefill_inputs(seed, L, T, d, dtype, threads=0):
    """i.i.d. N(0, I) hidden states [L, T, d]."""
    np_dt = np.float32 if dtype == F32 else np.uint16
    out = np.empty((L, T, d), dtype=np_dt)
    lib().wdg_prefill_inputs(seed, L, T, d, dtype, out.ctypes.data, threads)
    return out
