"""Device-side filling of synthetic tensors (same bits as the host generator).

Loads ``libkvp_inputs.so`` (built next to this file by
``python -m paper_2608_15943_amd.build``).  Used by the GPU tests and the
benchmark to materialise large weights, activations and caches in HBM without
a host round trip; the oracle regenerates what it needs with the host code in
``kvp_inputs``.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

from . import (KIND_DY, KIND_KCACHE, KIND_VCACHE, KIND_WK, KIND_WO, KIND_WQ, KIND_WV, KIND_X, KIND_XDEC,
               POS_STRIDE, Workload, normal_scale, stream_key, tensor_id, weight_shape)

_LIB = None
LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libkvp_inputs.so")


def _lib():
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run `python -m paper_2608_15943_amd.build`")
        L = C.CDLL(LIB_PATH)
        L.kvpin_fill.argtypes = [C.c_void_p, C.c_int, C.c_uint64, C.c_float,
                                 C.POINTER(C.c_int64), C.POINTER(C.c_int64), C.POINTER(C.c_uint64),
                                 C.c_void_p]
        L.kvpin_fill.restype = C.c_int
        L.kvpin_fill_pages.argtypes = [C.c_void_p, C.c_int, C.c_uint64, C.c_float, C.c_void_p, C.c_int,
                                       C.c_int, C.c_void_p, C.c_int, C.c_int, C.c_int, C.c_int,
                                       C.c_uint64, C.c_uint64, C.c_void_p]
        L.kvpin_fill_pages.restype = C.c_int
        _LIB = L
    return _LIB


def fill(ptr: int, dtype: str, seed: int, tid: int, sigma: float, dims, dst_strides, log_strides,
         stream: int = 0) -> None:
    """Fill a strided 4-d view: element (i0..i3) at sum(i_k * dst_strides[k]) gets the
    generator value of logical index sum(i_k * log_strides[k])."""
    dims = list(dims) + [1] * (4 - len(dims))
    ds = list(dst_strides) + [0] * (4 - len(dst_strides))
    ls = list(log_strides) + [0] * (4 - len(log_strides))
    kind = 0 if dtype == "bf16" else 1
    rc = _lib().kvpin_fill(C.c_void_p(ptr), kind, C.c_uint64(stream_key(seed, tid)),
                           C.c_float(float(normal_scale(sigma))), (C.c_int64 * 4)(*dims),
                           (C.c_int64 * 4)(*ds), (C.c_uint64 * 4)(*ls), C.c_void_p(stream or None))
    if rc != 0:
        raise RuntimeError(f"kvpin_fill failed ({rc})")


def fill_weight(w: Workload, kind: int, layer: int, ptr: int, stream: int = 0) -> None:
    rows, cols = weight_shape(w, kind)
    fill(ptr, w.dtype, w.seed, tensor_id(kind, layer), w.w_sigma, [rows, cols], [cols, 1],
         [cols, 1], stream)


def fill_prefill_x(w: Workload, ptr: int, B: int, S: int, stream: int = 0) -> None:
    """x [B, S, h] with the logical (b, pos, c) indexing of kvp_inputs.act_index."""
    fill(ptr, w.dtype, w.seed, tensor_id(KIND_X), w.x_sigma, [B, S, w.h],
         [S * w.h, w.h, 1], [POS_STRIDE * w.h, w.h, 1], stream)


def fill_prefill_dy(w: Workload, ptr: int, B: int, S: int, stream: int = 0) -> None:
    """dLoss/dY [B, S, h] in fp32, indexed like the prefill input."""
    fill(ptr, "fp32", w.seed, tensor_id(KIND_DY), 1.0, [B, S, w.h],
         [S * w.h, w.h, 1], [POS_STRIDE * w.h, w.h, 1], stream)


def fill_decode_x(w: Workload, ptr: int, B: int, stream: int = 0) -> None:
    fill(ptr, w.dtype, w.seed, tensor_id(KIND_XDEC), w.x_sigma, [B, w.h], [w.h, 1],
         [POS_STRIDE * w.h, 1], stream)


def fill_cache(w: Workload, layer: int, k_ptr: int, v_ptr: int, B: int, cap: int, npos: int,
               stream: int = 0) -> None:
    """Slots of producer ``layer``: K [B][g][cap][d] and V [B][g][d][cap]; positions [0, npos)."""
    g, d = w.g, w.d_h
    fill(k_ptr, w.dtype, w.seed, tensor_id(KIND_KCACHE, layer), w.cache_sigma, [B, g, npos, d],
         [g * cap * d, cap * d, d, 1], [g * POS_STRIDE * d, POS_STRIDE * d, d, 1], stream)
    fill(v_ptr, w.dtype, w.seed, tensor_id(KIND_VCACHE, layer), w.cache_sigma, [B, g, d, npos],
         [g * d * cap, d * cap, cap, 1], [g * POS_STRIDE * d, POS_STRIDE * d, 1, d], stream)


def fill_cache_pages(w: Workload, layer: int, k_pool: int, v_pool: int, pages_dev: int, stride: int,
                     n_pages: int, npos_dev: int, B: int, stream: int = 0) -> None:
    """Producer ``layer``'s page pools (K [g][n][64][d], V [g][n][d][64]) hold the same
    values as fill_cache's slots: position p < npos[b] of sequence b at page
    pages[b][p // 64], row p % 64 (device int32 arrays pages [B][stride], npos [B])."""
    g, d = w.g, w.d_h
    kind = 0 if w.dtype == "bf16" else 1
    sc = C.c_float(float(normal_scale(w.cache_sigma)))
    for tid, ptr, tr in ((tensor_id(KIND_KCACHE, layer), k_pool, 0), (tensor_id(KIND_VCACHE, layer), v_pool, 1)):
        rc = _lib().kvpin_fill_pages(C.c_void_p(ptr), kind, C.c_uint64(stream_key(w.seed, tid)), sc,
                                     C.c_void_p(pages_dev), stride, n_pages, C.c_void_p(npos_dev), B, g, d, tr,
                                     C.c_uint64(g * POS_STRIDE * d), C.c_uint64(POS_STRIDE * d),
                                     C.c_void_p(stream or None))
        if rc != 0:
            raise RuntimeError(f"kvpin_fill_pages failed ({rc})")


__all__ = ["fill", "fill_weight", "fill_prefill_x", "fill_decode_x", "fill_cache", "fill_cache_pages", "np"]
