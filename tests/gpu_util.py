"""Helpers for the GPU parity tests: build a model on the device through the C
ABI from a seeded workload, and the matching fp64 oracle inputs on the host.

Inputs on both sides come only from kvp_inputs (device filler and host
generator, bit-identical); the oracle never sees a value the HIP path made.
"""
from __future__ import annotations

import sys
from dataclasses import dataclass, field
from typing import Dict, List, Optional

import numpy as np
import torch

import kvp_inputs as ki
from kvp_inputs import device as kd
from oracle import attention as oat
from paper_2608_15943_amd import binding as kb

DEV = "cuda"


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def tdtype(w):
    return torch.bfloat16 if w.dtype == "bf16" else torch.float32


def kdtype(w):
    return kb.KVP_DTYPE_BF16 if w.dtype == "bf16" else kb.KVP_DTYPE_FP32


def tol(w):
    """max|err| <= tol * max|ref|: 2e-2 for bf16, 1e-5 for fp32."""
    return 2e-2 if w.dtype == "bf16" else 1e-5


def rel_err(got, ref):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    assert np.all(np.isfinite(got)), "non-finite values in the GPU result"
    return float(np.abs(got - ref).max() / max(np.abs(ref).max(), 1e-30))


def to_np(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


@dataclass
class DeviceModel:
    w: ki.Workload
    model: kb.Model
    B: int
    cap: int
    tensors: Dict[str, torch.Tensor] = field(default_factory=dict)
    slots: Dict[int, tuple] = field(default_factory=dict)


def build_device_model(w: ki.Workload, B: int, max_seq: int, cap: int,
                       fill_cache_npos: int = 0) -> DeviceModel:
    m = kb.Model(w.L, w.h, w.a, w.g, w.d_h, kdtype(w), w.tau, max_batch=B, max_seq=max_seq,
                 kv_capacity=cap, rope_base=w.rope_base)
    dm = DeviceModel(w, m, B, cap)
    dt = tdtype(w)
    for l in range(w.L):
        prod = w.tau[l] == l
        ts = {}
        for kind, name in ((ki.KIND_WQ, "wq"), (ki.KIND_WO, "wo")) + (
                ((ki.KIND_WK, "wk"), (ki.KIND_WV, "wv")) if prod else ()):
            rows, cols = ki.weight_shape(w, kind)
            t = torch.empty((rows, cols), dtype=dt, device=DEV)
            kd.fill_weight(w, kind, l, t.data_ptr())
            ts[name] = t
            dm.tensors[f"{name}{l}"] = t
        m.kvp_set_layer(l, ts["wq"].data_ptr(), ts["wk"].data_ptr() if prod else 0,
                        ts["wv"].data_ptr() if prod else 0, ts["wo"].data_ptr())
        if prod:
            K = torch.zeros((B, w.g, cap, w.d_h), dtype=dt, device=DEV)
            V = torch.zeros((B, w.g, w.d_h, cap), dtype=dt, device=DEV)
            if fill_cache_npos:
                kd.fill_cache(w, l, K.data_ptr(), V.data_ptr(), B, cap, fill_cache_npos)
            m.kvp_set_kv_slot(l, K.data_ptr(), V.data_ptr())
            dm.slots[l] = (K, V)
    torch.cuda.synchronize()
    return dm


def oracle_weights(w: ki.Workload) -> List[oat.LayerWeights]:
    out = []
    for l in range(w.L):
        prod = w.tau[l] == l
        out.append(oat.LayerWeights(
            ki.weight(w, ki.KIND_WQ, l),
            ki.weight(w, ki.KIND_WK, l) if prod else None,
            ki.weight(w, ki.KIND_WV, l) if prod else None,
            ki.weight(w, ki.KIND_WO, l)))
    return out


def workspace(dm: DeviceModel, phase: int, B: int, S: int = 1):
    n = dm.model.kvp_workspace_size(phase, B, S)
    ws = torch.empty(n, dtype=torch.uint8, device=DEV)
    return ws, n


def run_prefill(dm: DeviceModel, B: int, S: int):
    w = dm.w
    x = torch.empty((B, S, w.h), dtype=tdtype(w), device=DEV)
    kd.fill_prefill_x(w, x.data_ptr(), B, S)
    y = torch.empty_like(x)
    ws, n = workspace(dm, kb.KVP_PHASE_PREFILL, B, S)
    dm.model.kvp_prefill(x.data_ptr(), y.data_ptr(), B, S, ws.data_ptr(), n,
                         torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    return x, y


def small_workload(name, L, h, a, g, tau, dtype="bf16", d_h=128, seed=0):
    return ki.Workload(name=name, L=L, h=h, a=a, g=g, d_h=d_h, dtype=dtype, tau=list(tau),
                       phase="prefill", batch=1, seq=1, seed=seed)


def _align256(n: int) -> int:
    return (n + 255) // 256 * 256


def saved_views(w: ki.Workload, saved: torch.Tensor, B: int, S: int):
    """Per-layer views of kvp_train_forward's `saved` buffer (bf16 models), in the layout
    the C ABI documents: layer l at l * stride holds Q [B*S, a*d_h], O [B*S, a*d_h], the
    layer input X [B*S, h] (l >= 1), the row log-sum-exp [B, a, S rounded up to 64] and,
    when B*S % 512 == 0 and S % 8 == 0, O^T [a*d_h, B*S] (key "ot")."""
    M, nq = B * S, w.a * w.d_h
    q_off = 0
    o_off = q_off + _align256(M * nq * 2)
    x_off = o_off + _align256(M * nq * 2)
    lse_off = x_off + _align256(M * w.h * 2)
    ot_off = lse_off + _align256(B * w.a * ((S + 63) // 64 * 64) * 4)
    has_ot = M % 512 == 0 and S % 8 == 0
    stride = ot_off + (_align256(M * nq * 2) if has_ot else 0)
    assert stride * w.L == saved.numel(), (stride * w.L, saved.numel())
    out = []
    for l in range(w.L):
        base = l * stride
        v = {
            "q": saved[base + q_off: base + q_off + M * nq * 2].view(torch.bfloat16).view(B, S, nq),
            "o": saved[base + o_off: base + o_off + M * nq * 2].view(torch.bfloat16).view(B, S, nq),
            "x": saved[base + x_off: base + x_off + M * w.h * 2].view(torch.bfloat16).view(B, S, w.h),
        }
        if has_ot:
            v["ot"] = saved[base + ot_off: base + ot_off + M * nq * 2].view(torch.bfloat16).view(nq, M)
        out.append(v)
    return out
