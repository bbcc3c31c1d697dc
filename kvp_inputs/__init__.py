"""Seeded synthetic inputs shared by the oracle, the tests and the benchmark.

This module holds no attention or planner arithmetic. It only defines
(1) one counter-based random generator, (2) how each tensor of a workload is
named in that generator, and (3) the shapes and sharing maps of the workloads
the paper's experiments stand for (LLaMA2/LLaMA3/Qwen2.5-shaped attention
stacks, prefill at 4K-8K tokens and decode over 32K-128K-token caches).

Generator
---------
SplitMix64 (Steele, Lea and Flood, "Fast splittable pseudorandom number
generators", OOPSLA 2014): the n-th output of a stream with state ``key`` is
``mix64(key + n * GAMMA)`` with the published finaliser ``mix64``.  Element
``e`` of a tensor takes output ``n = e + 1`` of the tensor's stream.

Each 64-bit output is cut into four 16-bit integers ``u0..u3`` and turned into
an approximately normal value with the Irwin-Hall construction:

    z_num = (u0 + u1 + u2 + u3) - 131070          (an integer, |z_num| < 2**18)
    value = float32(z_num) * float32(sigma * sqrt(3) / 65536)

The product is one IEEE fp32 multiplication, so a device implementation of
the same steps gives the same bits.  The variance is sigma**2 * (1 - 2**-32).
bf16 tensors are the fp32 value rounded to nearest-even.

Every tensor is addressed by *logical* coordinates that do not depend on the
shape of the launch (row strides of 2**20 positions), so a prefix or a single
sequence of a large tensor can be regenerated on the host without producing
the rest.
"""
from __future__ import annotations

import math
import os
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence

import numpy as np

GAMMA = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)
_U16 = np.uint64(0xFFFF)

# Positions per sequence in the logical index space of activations and caches.
POS_STRIDE = 1 << 20

# Tensor kinds; the stream of tensor (kind, layer) is keyed by tensor_id().
KIND_X = 1        # prefill input activations [B, S, h]
KIND_WQ = 2       # query projection weight [a*d_h, h]
KIND_WK = 3       # key projection weight [g*d_h, h]
KIND_WV = 4       # value projection weight [g*d_h, h]
KIND_WO = 5       # output projection weight [h, a*d_h]
KIND_KCACHE = 6   # post-RoPE key cache contents, logical [B, g, pos, d_h]
KIND_VCACHE = 7   # value cache contents, logical [B, g, pos, d_h]
KIND_LENS = 8     # ragged decode context lengths [B]
KIND_XDEC = 9     # decode input activations [B, h]
KIND_DY = 10      # upstream gradient of the stack output [B, S, h] (always fp32)


def _mix64_inplace(z: np.ndarray) -> np.ndarray:
    """SplitMix64 finaliser applied in place to a uint64 array (wrapping arithmetic)."""
    t = np.empty_like(z)
    with np.errstate(over="ignore"):
        np.right_shift(z, np.uint64(30), out=t)
        z ^= t
        z *= _M1
        np.right_shift(z, np.uint64(27), out=t)
        z ^= t
        z *= _M2
        np.right_shift(z, np.uint64(31), out=t)
        z ^= t
    return z


def mix64(z: np.ndarray) -> np.ndarray:
    """SplitMix64 finaliser on a uint64 array (wrapping arithmetic)."""
    return _mix64_inplace(np.array(z, dtype=np.uint64, copy=True))


def tensor_id(kind: int, layer: int = 0) -> int:
    return (int(kind) << 16) | int(layer)


def stream_key(seed: int, tid: int) -> int:
    """64-bit stream state of tensor ``tid`` under ``seed``."""
    v = np.array([((int(seed) & 0xFFFFFFFF) << 32) | (int(tid) & 0xFFFFFFFF)],
                 dtype=np.uint64)
    return int(mix64(v)[0])


def raw64(key: int, idx: np.ndarray) -> np.ndarray:
    """Output idx+1 of the SplitMix64 stream with state ``key``."""
    z = np.array(idx, dtype=np.uint64, copy=True)
    with np.errstate(over="ignore"):
        z += np.uint64(1)
        z *= GAMMA
        z += np.uint64(key)
    return _mix64_inplace(z)


def normal_scale(sigma: float) -> np.float32:
    """fp32 constant that maps the Irwin-Hall numerator to N(0, sigma**2)."""
    return np.float32(float(sigma) * math.sqrt(3.0) / 65536.0)


def _normal_chunk(key: int, idx: np.ndarray, scale: np.float32, bf16: bool = False) -> np.ndarray:
    h = raw64(key, idx)
    s = (h & _U16).astype(np.int32)
    h >>= np.uint64(16)
    s += (h & _U16).astype(np.int32)
    h >>= np.uint64(16)
    s += (h & _U16).astype(np.int32)
    h >>= np.uint64(16)
    s += h.astype(np.int32)
    s -= 131070
    v = s.astype(np.float32) * scale
    return round_to_bf16(v) if bf16 else v


_CHUNK = 1 << 22


def normal_f32(key: int, idx: np.ndarray, sigma: float, bf16: bool = False) -> np.ndarray:
    """Irwin-Hall(4) normals at logical indices idx (any shape), optionally rounded to
    bf16 (returned as fp32); large inputs are split over threads."""
    idx = np.asarray(idx, dtype=np.uint64)
    scale = normal_scale(sigma)
    flat = idx.reshape(-1)
    n = flat.size
    if n <= _CHUNK:
        return _normal_chunk(key, flat, scale, bf16).reshape(idx.shape)
    out = np.empty(n, dtype=np.float32)

    def work(lo):
        hi = min(lo + _CHUNK, n)
        out[lo:hi] = _normal_chunk(key, flat[lo:hi], scale, bf16)

    import concurrent.futures as cf
    workers = max(1, min(16, os.cpu_count() or 1))
    with cf.ThreadPoolExecutor(workers) as ex:
        list(ex.map(work, range(0, n, _CHUNK)))
    return out.reshape(idx.shape)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round finite fp32 to bf16 (nearest-even) and return the 16-bit patterns."""
    u = np.array(x, dtype=np.float32, copy=True).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    u += np.uint32(0x7FFF)          # finite inputs stay below 2**32
    u += lsb
    u >>= np.uint32(16)
    return u.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """fp32 values rounded to the nearest bf16 value, returned as fp32."""
    return bf16_bits_to_f32(f32_to_bf16_bits(x))


def normal_values(seed: int, tid: int, idx: np.ndarray, sigma: float, dtype: str) -> np.ndarray:
    """Synthetic values at logical indices ``idx`` as fp32 (bf16-exact if dtype='bf16')."""
    if dtype not in ("bf16", "fp32"):
        raise ValueError(f"unknown dtype {dtype!r}")
    return normal_f32(stream_key(seed, tid), idx, sigma, bf16=(dtype == "bf16"))


# ---------------------------------------------------------------------------
# Logical index maps: one per tensor family.
# ---------------------------------------------------------------------------

def weight_index(rows: int, cols: int, row0: int = 0, nrows: Optional[int] = None) -> np.ndarray:
    nrows = rows - row0 if nrows is None else nrows
    r = np.arange(row0, row0 + nrows, dtype=np.uint64)[:, None]
    c = np.arange(cols, dtype=np.uint64)[None, :]
    return r * np.uint64(cols) + c


def act_index(batch_ids: Sequence[int], positions: Sequence[int], width: int) -> np.ndarray:
    """Logical index of activation rows (b, pos) -> [len(b), len(pos), width]."""
    b = np.asarray(batch_ids, dtype=np.uint64)[:, None, None]
    p = np.asarray(positions, dtype=np.uint64)[None, :, None]
    c = np.arange(width, dtype=np.uint64)[None, None, :]
    return (b * np.uint64(POS_STRIDE) + p) * np.uint64(width) + c


def cache_index(b: int, n_kv: int, positions: Sequence[int], d_h: int) -> np.ndarray:
    """Logical index of one sequence's cache, all kv heads -> [n_kv, len(pos), d_h]."""
    g = np.arange(n_kv, dtype=np.uint64)[:, None, None]
    p = np.asarray(positions, dtype=np.uint64)[None, :, None]
    d = np.arange(d_h, dtype=np.uint64)[None, None, :]
    return ((np.uint64(b) * np.uint64(n_kv) + g) * np.uint64(POS_STRIDE) + p) * np.uint64(d_h) + d


def ragged_lengths(seed: int, batch: int, lo: int, hi: int) -> np.ndarray:
    """Integer lengths uniform on {lo, ..., hi} (hi - lo + 1 must be a power of two <= 2**16)."""
    span = hi - lo + 1
    if span <= 0 or span > (1 << 16) or (span & (span - 1)):
        raise ValueError("length span must be a power of two up to 65536")
    h = raw64(stream_key(seed, tensor_id(KIND_LENS)), np.arange(batch, dtype=np.uint64))
    return (lo + ((h >> np.uint64(48)) & np.uint64(span - 1)).astype(np.int64)).astype(np.int32)


# ---------------------------------------------------------------------------
# Workloads.
# ---------------------------------------------------------------------------

@dataclass
class Workload:
    name: str
    L: int
    h: int
    a: int
    g: int
    d_h: int
    dtype: str
    tau: List[int]
    phase: str                      # "prefill" or "decode"
    batch: int
    seq: int = 0                    # prefill length
    ctx: int = 0                    # decode: context length (uniform) ...
    ctx_lo: int = 0                 # ... or ragged range [ctx_lo, ctx_hi]
    ctx_hi: int = 0
    kv_capacity: int = 0
    rope_base: float = 10000.0
    w_sigma: float = 0.02
    x_sigma: float = 1.0
    cache_sigma: float = 1.0
    seed: int = 0
    notes: str = ""
    extra: Dict[str, object] = field(default_factory=dict)

    def lengths(self) -> np.ndarray:
        if self.phase != "decode":
            raise ValueError("lengths are defined for decode workloads")
        if self.ctx_hi:
            return ragged_lengths(self.seed, self.batch, self.ctx_lo, self.ctx_hi)
        return np.full(self.batch, self.ctx, dtype=np.int32)

    def producers(self) -> List[int]:
        return [l for l in range(self.L) if self.tau[l] == l]

    def with_map(self, tau: Sequence[int], name_suffix: str = "") -> "Workload":
        import dataclasses
        return dataclasses.replace(self, tau=list(tau), name=self.name + name_suffix)


def _round_up(x: int, m: int) -> int:
    return (x + m - 1) // m * m


def tiny_fp32() -> Workload:
    return Workload(name="tiny-fp32-4L-d256-s128", L=4, h=256, a=4, g=4, d_h=64, dtype="fp32",
                    tau=[0, 0, 2, 2], phase="prefill", batch=1, seq=128, kv_capacity=128)


def stage_share_prefill() -> Workload:
    """One PP-stage share of a Llama-style model: 8 layers, d=2048, GQA 16/8 x 128, S=4096, B=4."""
    return Workload(name="prefill-8L-d2048-gqa16x8-s4096-b4", L=8, h=2048, a=16, g=8, d_h=128,
                    dtype="bf16", tau=[0, 1, 2, 3, 4, 4, 6, 6], phase="prefill", batch=4,
                    seq=4096, kv_capacity=4096)


def decode_32k() -> Workload:
    """32-layer d=4096 GQA 32/8 x 128, batch 64, 32768-token caches, odd layers share."""
    tau = [l - (l % 2) for l in range(32)]
    return Workload(name="decode-32L-d4096-gqa32x8-b64-ctx32k", L=32, h=4096, a=32, g=8, d_h=128,
                    dtype="bf16", tau=tau, phase="decode", batch=64, ctx=32768,
                    kv_capacity=_round_up(32768 + 1, 64))


def decode_128k_ragged() -> Workload:
    """Same model, batch 8, ragged 64K-128K contexts, groups of 4 layers share their first."""
    tau = [l - (l % 4) for l in range(32)]
    return Workload(name="decode-32L-d4096-gqa32x8-b8-ctx64k-128k", L=32, h=4096, a=32, g=8,
                    d_h=128, dtype="bf16", tau=tau, phase="decode", batch=8,
                    ctx_lo=65536, ctx_hi=131071, kv_capacity=131072)


def stage_70b_prefill(tau: Optional[Sequence[int]] = None) -> Workload:
    """70B-shaped PP=8 stage on one GPU: 10 layers, d=8192, GQA 64/8 x 128, S=8192, B=1.

    The sharing map comes from the FIR rule; the planner run that produces it
    lives with the caller (tests and bench), the default here is its result.
    """
    return Workload(name="prefill-10L-d8192-gqa64x8-s8192-b1", L=10, h=8192, a=64, g=8, d_h=128,
                    dtype="bf16", tau=list(tau) if tau is not None else [0] * 10,
                    phase="prefill", batch=1, seq=8192, kv_capacity=8192)


WORKLOADS = {
    "tiny": tiny_fp32,
    "prefill": stage_share_prefill,
    "decode": decode_32k,
    "decode_long": decode_128k_ragged,
    "prefill_70b": stage_70b_prefill,
}


# ---------------------------------------------------------------------------
# Host-side materialisation (used by the oracle side; the device fills its own).
# ---------------------------------------------------------------------------

def weight(w: Workload, kind: int, layer: int, row0: int = 0, nrows: Optional[int] = None) -> np.ndarray:
    rows, cols = weight_shape(w, kind)
    idx = weight_index(rows, cols, row0, nrows)
    return normal_values(w.seed, tensor_id(kind, layer), idx, w.w_sigma, w.dtype)


def weight_shape(w: Workload, kind: int):
    if kind == KIND_WQ:
        return w.a * w.d_h, w.h
    if kind in (KIND_WK, KIND_WV):
        return w.g * w.d_h, w.h
    if kind == KIND_WO:
        return w.h, w.a * w.d_h
    raise ValueError(kind)


def prefill_x(w: Workload, batch_ids: Sequence[int], positions: Sequence[int]) -> np.ndarray:
    idx = act_index(batch_ids, positions, w.h)
    return normal_values(w.seed, tensor_id(KIND_X), idx, w.x_sigma, w.dtype)


def prefill_dy(w: Workload, batch_ids: Sequence[int], positions: Sequence[int]) -> np.ndarray:
    """dLoss/dY rows (b, pos) -> [len(b), len(pos), h], fp32, standard normal."""
    idx = act_index(batch_ids, positions, w.h)
    return normal_values(w.seed, tensor_id(KIND_DY), idx, 1.0, "fp32")


def decode_x(w: Workload, batch_ids: Sequence[int]) -> np.ndarray:
    idx = act_index(batch_ids, [0], w.h)[:, 0, :]
    return normal_values(w.seed, tensor_id(KIND_XDEC), idx, w.x_sigma, w.dtype)


def cache_contents(w: Workload, kind: int, layer: int, b: int, length: int) -> np.ndarray:
    """Synthetic post-RoPE K (kind=KIND_KCACHE) or V of one sequence: [g, length, d_h]."""
    idx = cache_index(b, w.g, np.arange(length), w.d_h)
    return normal_values(w.seed, tensor_id(kind, layer), idx, w.cache_sigma, w.dtype)
