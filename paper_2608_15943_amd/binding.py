"""ctypes binding of the C ABI in include/kvpipe.h (argument marshalling only).

Every function keeps the C name.  Device buffers are passed as integer
addresses (``tensor.data_ptr()``), streams as the raw hipStream_t
(``torch.cuda.current_stream().cuda_stream``).  Non-zero status codes raise
KvpError carrying the code and kvp_last_error().  Nothing here computes: if
the library is missing the first call raises, there is no fallback.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np
from typing import Optional, Sequence

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "lib", "libkvpipe.so")

KVP_OK = 0
KVP_E_INVALID_ARG = -1
KVP_E_BAD_MAP = -2
KVP_E_SHAPE = -3
KVP_E_WORKSPACE = -4
KVP_E_CAPACITY = -5
KVP_E_HIP = -6
KVP_E_STATE = -7

KVP_DTYPE_BF16 = 0
KVP_DTYPE_FP32 = 1
KVP_PHASE_PREFILL = 0
KVP_PHASE_DECODE = 1
KVP_PHASE_BACKWARD = 2
KVP_STOP_FIR_MET = 0
KVP_STOP_BUDGET = 1
KVP_STOP_NO_CONVERTIBLE = 2
KVP_PLACE_UNIFORM = 0
KVP_PLACE_SYMMETRIC_BIPOLAR = 1

EXPORTS = [
    "kvp_layer_flops", "kvp_fir", "kvp_plan_fir", "kvp_stage_flops", "kvp_place",
    "kvp_map_from_mask", "kvp_canonicalize_map",
    "kvp_create", "kvp_destroy", "kvp_set_layer", "kvp_set_kv_slot", "kvp_workspace_size",
    "kvp_prefill", "kvp_layer_forward", "kvp_decode_step", "kvp_get_map", "kvp_status_string",
    "kvp_last_error", "kvp_profile_enable", "kvp_profile_read",
    "kvp_train_saved_size", "kvp_train_forward", "kvp_set_layer_grads", "kvp_backward",
    "kvp_set_kv_pool", "kvp_page_bytes", "kvp_prefill_paged", "kvp_decode_step_paged",
    "kvp_pager_create", "kvp_pager_destroy", "kvp_pager_reserve", "kvp_pager_release",
    "kvp_pager_free_pages", "kvp_pager_rows", "kvp_decode_step_noalloc",
    # include/kvp_calib.h: achievable-peak calibration (measurement support)
    "kvp_calib_mfma_bf16", "kvp_calib_stream_read",
]

KERNEL_KINDS = ["rope_table", "qkv_gemm", "flash_attn", "oproj_gemm", "dec_gemm", "dec_rope",
                "dec_attn", "dec_combine", "dec_oproj", "f32_rope", "f32_attn", "bwd_gemm",
                "bwd_attn_kv", "bwd_attn_q", "bwd_aux"]


class kvp_shape(C.Structure):
    _fields_ = [("b", C.c_int64), ("s", C.c_int64), ("h", C.c_int64), ("a", C.c_int64),
                ("g", C.c_int64), ("ffn", C.c_int64), ("causal", C.c_int32), ("_pad", C.c_int32)]


class kvp_plan_in(C.Structure):
    _fields_ = [("L", C.c_int32), ("P", C.c_int32), ("stage_of_layer", C.POINTER(C.c_int32)),
                ("f_full", C.POINTER(C.c_double)), ("f_share", C.POINTER(C.c_double)),
                ("f_lmhead", C.c_double), ("eps", C.c_double), ("m", C.c_int32),
                ("_pad", C.c_int32), ("admissible", C.POINTER(C.c_uint8)), ("alpha", C.c_double)]


class kvp_plan_out(C.Structure):
    _fields_ = [("z", C.POINTER(C.c_uint8)), ("stage_flops", C.POINTER(C.c_double)),
                ("fir", C.c_double), ("n_converted", C.c_int32), ("stop_reason", C.c_int32)]


class kvp_model_desc(C.Structure):
    _fields_ = [("L", C.c_int32), ("h", C.c_int32), ("a", C.c_int32), ("g", C.c_int32),
                ("d_h", C.c_int32), ("dtype", C.c_int32), ("rope_base", C.c_double),
                ("max_batch", C.c_int32), ("max_seq", C.c_int32), ("kv_capacity", C.c_int32),
                ("_pad", C.c_int32)]


class KvpError(RuntimeError):
    def __init__(self, code: int, where: str, msg: str):
        super().__init__(f"{where}: {status_name(code)} ({code}): {msg}")
        self.code = code


_lib: Optional[C.CDLL] = None


def lib() -> C.CDLL:
    """Load libkvpipe.so (built by paper_2608_15943_amd.build); raise if absent."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built; run `python -m paper_2608_15943_amd.build`")
    L = C.CDLL(LIB_PATH)
    vp, i32, i64, dbl = C.c_void_p, C.c_int, C.c_int64, C.c_double
    sig = {
        "kvp_layer_flops": ([C.POINTER(kvp_shape), i32, C.POINTER(dbl), C.POINTER(dbl)], i32),
        "kvp_fir": ([i32, C.POINTER(dbl), C.POINTER(dbl)], i32),
        "kvp_plan_fir": ([C.POINTER(kvp_plan_in), C.POINTER(kvp_plan_out)], i32),
        "kvp_stage_flops": ([i32, i32, C.POINTER(C.c_int32), C.POINTER(dbl), C.POINTER(dbl),
                             C.POINTER(C.c_uint8), dbl, C.POINTER(dbl)], i32),
        "kvp_place": ([i32, i32, i32, C.POINTER(C.c_int32), i32, C.POINTER(C.c_uint8), dbl,
                       C.POINTER(C.c_uint8), C.POINTER(C.c_int32), C.POINTER(C.c_int32)], i32),
        "kvp_map_from_mask": ([i32, C.POINTER(C.c_uint8), C.POINTER(C.c_int32)], i32),
        "kvp_canonicalize_map": ([i32, C.POINTER(C.c_int32), C.POINTER(C.c_int32)], i32),
        "kvp_create": ([C.POINTER(kvp_model_desc), C.POINTER(C.c_int32), C.POINTER(vp)], i32),
        "kvp_destroy": ([vp], i32),
        "kvp_set_layer": ([vp, i32, vp, vp, vp, vp], i32),
        "kvp_set_kv_slot": ([vp, i32, vp, vp], i32),
        "kvp_workspace_size": ([vp, i32, i32, i32, C.POINTER(C.c_size_t)], i32),
        "kvp_prefill": ([vp, vp, vp, i32, i32, vp, C.c_size_t, vp], i32),
        "kvp_layer_forward": ([vp, i32, vp, vp, vp, i32, i32, vp, C.c_size_t, vp], i32),
        "kvp_decode_step": ([vp, vp, vp, i32, vp, i32, vp, C.c_size_t, vp], i32),
        "kvp_get_map": ([vp, C.POINTER(C.c_int32)], i32),
        "kvp_train_saved_size": ([vp, i32, i32, C.POINTER(C.c_size_t)], i32),
        "kvp_train_forward": ([vp, vp, vp, i32, i32, vp, C.c_size_t, vp, C.c_size_t, vp], i32),
        "kvp_set_layer_grads": ([vp, i32, vp, vp, vp, vp], i32),
        "kvp_backward": ([vp, vp, vp, vp, i32, i32, vp, C.c_size_t, vp, C.c_size_t, vp], i32),
        "kvp_set_kv_pool": ([vp, i32, vp, vp, i32], i32),
        "kvp_page_bytes": ([vp, C.POINTER(C.c_size_t)], i32),
        "kvp_prefill_paged": ([vp, vp, vp, i32, i32, vp, i32, vp, C.c_size_t, vp], i32),
        "kvp_decode_step_paged": ([vp, vp, vp, i32, vp, i32, vp, i32, vp, C.c_size_t, vp], i32),
        "kvp_decode_step_noalloc": ([vp, vp, vp, i32, vp, i32, vp], i32),
        "kvp_pager_create": ([i32, i32, i32, C.POINTER(vp)], i32),
        "kvp_pager_destroy": ([vp], None),
        "kvp_pager_reserve": ([vp, i32, i32], i32),
        "kvp_pager_release": ([vp, i32], i32),
        "kvp_pager_free_pages": ([vp, C.POINTER(i32)], i32),
        "kvp_pager_rows": ([vp, C.POINTER(C.c_int32), i32, C.POINTER(C.c_int32)], i32),
        "kvp_status_string": ([i32], C.c_char_p),
        "kvp_last_error": ([], C.c_char_p),
        "kvp_profile_enable": ([vp, i32], i32),
        "kvp_profile_read": ([vp, C.POINTER(dbl), C.POINTER(i64)], i32),
        "kvp_calib_mfma_bf16": ([i32, vp, C.POINTER(dbl), vp], i32),
        "kvp_calib_stream_read": ([vp, C.c_size_t, vp, vp], i32),
    }
    for name, (args, res) in sig.items():
        fn = getattr(L, name)
        fn.argtypes = args
        fn.restype = res
    _lib = L
    return L


def status_name(code: int) -> str:
    try:
        return lib().kvp_status_string(code).decode()
    except Exception:
        return str(code)


def _check(code: int, where: str) -> None:
    if code != KVP_OK:
        raise KvpError(code, where, lib().kvp_last_error().decode())


def _i32(xs: Sequence[int]):
    return (C.c_int32 * len(xs))(*[int(x) for x in xs])


def _f64(xs: Sequence[float]):
    return (C.c_double * len(xs))(*[float(x) for x in xs])


# ---- planner -----------------------------------------------------------------

def kvp_layer_flops(b, s, h, a, g, ffn=0, causal=True, phase=KVP_PHASE_PREFILL):
    sh = kvp_shape(b, s, h, a, g, ffn, 1 if causal else 0, 0)
    f0, f1 = C.c_double(), C.c_double()
    _check(lib().kvp_layer_flops(C.byref(sh), phase, C.byref(f0), C.byref(f1)), "kvp_layer_flops")
    return f0.value, f1.value


def kvp_fir(stage_flops: Sequence[float]) -> float:
    out = C.c_double()
    _check(lib().kvp_fir(len(stage_flops), _f64(stage_flops), C.byref(out)), "kvp_fir")
    return out.value


def kvp_plan_fir(stage_of_layer, f_full, f_share, f_lmhead, eps, m=0, admissible=None, alpha=-1.0,
                 P=None):
    """Algorithm 1; returns dict(z, stage_flops, fir, n_converted, stop_reason)."""
    L = len(stage_of_layer)
    P = (max(stage_of_layer) + 1) if P is None else P
    adm = None
    if admissible is not None:
        adm = (C.c_uint8 * L)(*[1 if x else 0 for x in admissible])
    pin = kvp_plan_in(L, P, _i32(stage_of_layer), _f64(f_full), _f64(f_share), float(f_lmhead),
                      float(eps), int(m), 0,
                      C.cast(adm, C.POINTER(C.c_uint8)) if adm is not None else None, float(alpha))
    z = (C.c_uint8 * L)()
    F = (C.c_double * P)()
    pout = kvp_plan_out(C.cast(z, C.POINTER(C.c_uint8)), C.cast(F, C.POINTER(C.c_double)), 0.0, 0, 0)
    _check(lib().kvp_plan_fir(C.byref(pin), C.byref(pout)), "kvp_plan_fir")
    return dict(z=list(z), stage_flops=list(F), fir=pout.fir, n_converted=pout.n_converted,
                stop_reason=pout.stop_reason)


def kvp_stage_flops(stage_of_layer, f_full, f_share, z, f_lmhead, P=None):
    """Eq. (stage_flops_z): per-stage FLOPs of a mask, LM head on the last stage."""
    L = len(stage_of_layer)
    P = (max(stage_of_layer) + 1) if P is None else P
    F = (C.c_double * P)()
    _check(lib().kvp_stage_flops(L, P, _i32(stage_of_layer), _f64(f_full), _f64(f_share),
                                 (C.c_uint8 * L)(*[1 if x else 0 for x in z]), float(f_lmhead), F),
           "kvp_stage_flops")
    return list(F)


def kvp_place(strategy, stage_of_layer, k, admissible=None, alpha=-1.0, P=None):
    """Sec. 2.5 Uniform / Symmetric Bipolar placement; returns (z, n_placed, stop_reason)."""
    L = len(stage_of_layer)
    P = (max(stage_of_layer) + 1) if P is None else P
    adm = None if admissible is None else (C.c_uint8 * L)(*[1 if x else 0 for x in admissible])
    z = (C.c_uint8 * L)()
    n, stop = C.c_int32(), C.c_int32()
    _check(lib().kvp_place(int(strategy), L, P, _i32(stage_of_layer), int(k), adm, float(alpha), z,
                           C.byref(n), C.byref(stop)), "kvp_place")
    return list(z), n.value, stop.value


def kvp_map_from_mask(z: Sequence[int]):
    L = len(z)
    tau = (C.c_int32 * L)()
    _check(lib().kvp_map_from_mask(L, (C.c_uint8 * L)(*[int(x) for x in z]), tau), "kvp_map_from_mask")
    return list(tau)


def kvp_canonicalize_map(tau_in: Sequence[int]):
    L = len(tau_in)
    out = (C.c_int32 * L)()
    _check(lib().kvp_canonicalize_map(L, _i32(tau_in), out), "kvp_canonicalize_map")
    return list(out)


# ---- attention stack -------------------------------------------------------------

class Model:
    """Owns a kvp_ctx; device pointers are plain integers."""

    def __init__(self, L, h, a, g, d_h, dtype, tau, max_batch, max_seq, kv_capacity,
                 rope_base=10000.0):
        desc = kvp_model_desc(L, h, a, g, d_h, dtype, float(rope_base), max_batch, max_seq,
                              kv_capacity, 0)
        ctx = C.c_void_p()
        _check(lib().kvp_create(C.byref(desc), _i32(tau), C.byref(ctx)), "kvp_create")
        self.ctx = ctx
        self.L = L

    def close(self):
        if self.ctx:
            lib().kvp_destroy(self.ctx)
            self.ctx = C.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def kvp_set_layer(self, l, wq, wk, wv, wo):
        _check(lib().kvp_set_layer(self.ctx, l, wq, wk or None, wv or None, wo), "kvp_set_layer")

    def kvp_set_kv_slot(self, l, k, v):
        _check(lib().kvp_set_kv_slot(self.ctx, l, k, v), "kvp_set_kv_slot")

    def kvp_workspace_size(self, phase, B, S=1) -> int:
        n = C.c_size_t()
        _check(lib().kvp_workspace_size(self.ctx, phase, B, S, C.byref(n)), "kvp_workspace_size")
        return n.value

    def kvp_prefill(self, x, y, B, S, ws, ws_bytes, stream=0):
        _check(lib().kvp_prefill(self.ctx, x, y, B, S, ws, ws_bytes, stream or None), "kvp_prefill")

    def kvp_layer_forward(self, l, x, attn_out, y, B, S, ws, ws_bytes, stream=0):
        _check(lib().kvp_layer_forward(self.ctx, l, x, attn_out or None, y, B, S, ws, ws_bytes,
                                       stream or None), "kvp_layer_forward")

    def kvp_train_saved_size(self, B, S) -> int:
        n = C.c_size_t()
        _check(lib().kvp_train_saved_size(self.ctx, B, S, C.byref(n)), "kvp_train_saved_size")
        return n.value

    def kvp_train_forward(self, x, y, B, S, saved, saved_bytes, ws, ws_bytes, stream=0):
        _check(lib().kvp_train_forward(self.ctx, x, y, B, S, saved, saved_bytes, ws, ws_bytes,
                                       stream or None), "kvp_train_forward")

    def kvp_set_layer_grads(self, l, dwq, dwk, dwv, dwo):
        _check(lib().kvp_set_layer_grads(self.ctx, l, dwq or None, dwk or None, dwv or None,
                                         dwo or None), "kvp_set_layer_grads")

    def kvp_backward(self, x, dy, dx, B, S, saved, saved_bytes, ws, ws_bytes, stream=0):
        _check(lib().kvp_backward(self.ctx, x, dy, dx, B, S, saved, saved_bytes, ws, ws_bytes,
                                  stream or None), "kvp_backward")

    def kvp_decode_step(self, x, len_dev, max_len, y, B, ws, ws_bytes, stream=0):
        _check(lib().kvp_decode_step(self.ctx, x, len_dev, max_len, y, B, ws, ws_bytes,
                                     stream or None), "kvp_decode_step")

    def kvp_decode_step_noalloc(self, x, len_dev, max_len, y, B, stream=0):
        _check(lib().kvp_decode_step_noalloc(self.ctx, x, len_dev, max_len, y, B, stream or None),
               "kvp_decode_step_noalloc")

    def kvp_set_kv_pool(self, l, k, v, n_pages):
        _check(lib().kvp_set_kv_pool(self.ctx, l, k, v, n_pages), "kvp_set_kv_pool")

    def kvp_page_bytes(self) -> int:
        n = C.c_size_t()
        _check(lib().kvp_page_bytes(self.ctx, C.byref(n)), "kvp_page_bytes")
        return n.value

    def kvp_prefill_paged(self, x, y, B, S, pages_dev, pages_stride, ws, ws_bytes, stream=0):
        _check(lib().kvp_prefill_paged(self.ctx, x, y, B, S, pages_dev, pages_stride, ws, ws_bytes,
                                       stream or None), "kvp_prefill_paged")

    def kvp_decode_step_paged(self, x, len_dev, max_len, pages_dev, pages_stride, y, B, ws, ws_bytes,
                              stream=0):
        _check(lib().kvp_decode_step_paged(self.ctx, x, len_dev, max_len, pages_dev, pages_stride, y, B,
                                           ws, ws_bytes, stream or None), "kvp_decode_step_paged")

    def kvp_profile_enable(self, enable=True):
        _check(lib().kvp_profile_enable(self.ctx, 1 if enable else 0), "kvp_profile_enable")

    def kvp_profile_read(self):
        """{kind: (launches, total_ms)} for the launches timed since the last read."""
        n = len(KERNEL_KINDS)
        ms = (C.c_double * n)()
        cnt = (C.c_int64 * n)()
        _check(lib().kvp_profile_read(self.ctx, ms, cnt), "kvp_profile_read")
        return {KERNEL_KINDS[k]: (cnt[k], ms[k]) for k in range(n) if cnt[k]}

    def kvp_get_map(self):
        tau = (C.c_int32 * self.L)()
        _check(lib().kvp_get_map(self.ctx, tau), "kvp_get_map")
        return list(tau)


# ---- achievable-peak calibration (include/kvp_calib.h) ---------------------------------

def kvp_calib_mfma_bf16(iters: int, sink: int, stream: int = 0) -> float:
    """Launch the bf16 matrix-core loop; returns the launch's floating-point operations."""
    flops = C.c_double()
    _check(lib().kvp_calib_mfma_bf16(int(iters), C.c_void_p(sink), C.byref(flops), C.c_void_p(stream)),
           "kvp_calib_mfma_bf16")
    return flops.value


def kvp_calib_stream_read(src: int, nbytes: int, sink: int, stream: int = 0) -> None:
    """Launch the streaming read of nbytes at device address src."""
    _check(lib().kvp_calib_stream_read(C.c_void_p(src), C.c_size_t(nbytes), C.c_void_p(sink),
                                       C.c_void_p(stream)), "kvp_calib_stream_read")


class Pager:
    """Host page allocator (kvp_pager_*): a table of max_seqs rows x max_pages entries."""

    def __init__(self, n_pages, max_seqs, max_pages):
        p = C.c_void_p()
        _check(lib().kvp_pager_create(n_pages, max_seqs, max_pages, C.byref(p)), "kvp_pager_create")
        self.p = p
        self.max_pages = max_pages

    def close(self):
        if self.p:
            lib().kvp_pager_destroy(self.p)
            self.p = C.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def reserve(self, seq, n_tokens):
        _check(lib().kvp_pager_reserve(self.p, seq, n_tokens), "kvp_pager_reserve")

    def try_reserve(self, seq, n_tokens) -> bool:
        """reserve(); False (and nothing reserved) when the pool or the row is too small."""
        rc = lib().kvp_pager_reserve(self.p, seq, n_tokens)
        if rc == KVP_E_CAPACITY:
            return False
        _check(rc, "kvp_pager_reserve")
        return True

    def release(self, seq):
        _check(lib().kvp_pager_release(self.p, seq), "kvp_pager_release")

    def free_pages(self) -> int:
        n = C.c_int()
        _check(lib().kvp_pager_free_pages(self.p, C.byref(n)), "kvp_pager_free_pages")
        return n.value

    def rows(self, seqs):
        """Host table rows of seqs: numpy int32 [len(seqs)][max_pages], -1 where unmapped."""
        seqs = np.ascontiguousarray(seqs, dtype=np.int32)
        out = np.empty((len(seqs), self.max_pages), dtype=np.int32)
        _check(lib().kvp_pager_rows(self.p, seqs.ctypes.data_as(C.POINTER(C.c_int32)), len(seqs),
                                    out.ctypes.data_as(C.POINTER(C.c_int32))), "kvp_pager_rows")
        return out
