"""A precision model of the bf16 training forward, for bounding what the backward of a
deep bf16 stack can match (test infrastructure; CPU only).

The bf16 path rounds the forward activations it keeps to bf16: the projection input
X_l, the post-RoPE Q, K, V and the attention output O (the residual stream between layers
stays fp32).  The backward then differentiates at those rounded points.  This model runs
the oracle's arithmetic in fp64 with exactly those roundings (fp64 -> fp32 -> bf16, round
to nearest even) and is otherwise exact, so its distance from the exact oracle is the part
of the gradient error that no bf16 backward can remove.  It is built from the oracle's own
steps (projection, attention, their transposes) and shares nothing with the HIP path.
"""
from __future__ import annotations

from typing import Dict, List, Sequence, Tuple

import numpy as np

import kvp_inputs as ki
from oracle import attention as at
from oracle import backward as bw


def bf16(x: np.ndarray) -> np.ndarray:
    return ki.round_to_bf16(np.asarray(x, dtype=np.float64).astype(np.float32)).astype(np.float64)


def stack_backward_bf16_forward(x: np.ndarray, weights: Sequence[at.LayerWeights], tau: Sequence[int],
                                a: int, g: int, d_h: int, base: float, dy: np.ndarray):
    """stack_backward of the oracle with the forward activations rounded as the bf16 path keeps
    them.  Returns (dx [S, h], grads) like ``oracle.backward.stack_backward``."""
    S = x.shape[0]
    pos = np.arange(S)
    L = len(weights)
    xs, qs, os_ = [], [], []
    kv: Dict[int, Tuple[np.ndarray, np.ndarray]] = {}
    cur = np.asarray(x, dtype=np.float64)
    for l, w in enumerate(weights):
        xb = bf16(cur)
        xs.append(xb)
        prod = int(tau[l]) == l
        q, k, v = at.project_qkv(xb, pos, w, a, g, d_h, base, kv=prod)
        q = bf16(q)
        if prod:
            kv[l] = (bf16(k), bf16(v))
        k, v = kv[int(tau[l])]
        o = bf16(at._merge(at.attention(q, k, v, pos, pos)))
        qs.append(q)
        os_.append(o)
        cur = at.output_projection(cur, o, w)
    grads: List[dict] = [None] * L
    dk_acc: Dict[int, np.ndarray] = {}
    dv_acc: Dict[int, np.ndarray] = {}
    gx = np.asarray(dy, dtype=np.float64)
    for l in range(L - 1, -1, -1):
        w = weights[l]
        p = int(tau[l])
        dwo = gx.T @ os_[l]
        do = at._heads(gx @ w.wo, a, d_h)
        k, v = kv[p]
        dq, dk, dv = bw.attention_backward(qs[l], k, v, do, pos, pos)
        dk_acc[p] = dk_acc.get(p, 0.0) + dk
        dv_acc[p] = dv_acc.get(p, 0.0) + dv
        dq_pre = at._merge(bw.apply_rope_transpose(dq, pos, base))
        gnew = gx + dq_pre @ w.wq
        gr = {"dwq": dq_pre.T @ xs[l], "dwo": dwo, "dwk": None, "dwv": None}
        if p == l:
            dk_pre = at._merge(bw.apply_rope_transpose(dk_acc.pop(l), pos, base))
            dv_all = at._merge(dv_acc.pop(l))
            gr["dwk"] = dk_pre.T @ xs[l]
            gr["dwv"] = dv_all.T @ xs[l]
            gnew = gnew + dk_pre @ w.wk + dv_all @ w.wv
        grads[l] = gr
        gx = gnew
    return gx, grads


def stage_share_prefix_gradients(P: int = 300, batch: int = 4, kinds=("exact", "bf16")):
    """dX and the weight gradients (summed over the batch) of the 8-layer stage share on its
    first P positions, dY = the workload's seeded dY on those positions, for each of `kinds`:
    "exact" (the oracle) and "bf16" (the bf16-forward model).  Returns one (dx list, grads)
    per kind."""
    w = ki.stage_share_prefill()
    wts = [at.LayerWeights(ki.weight(w, ki.KIND_WQ, l),
                           ki.weight(w, ki.KIND_WK, l) if w.tau[l] == l else None,
                           ki.weight(w, ki.KIND_WV, l) if w.tau[l] == l else None,
                           ki.weight(w, ki.KIND_WO, l)) for l in range(w.L)]
    out = []
    fns = {"exact": bw.stack_backward, "bf16": stack_backward_bf16_forward}
    for fn in (fns[k] for k in kinds):
        dxs, tot = [], None
        for b in range(batch):
            xb = ki.prefill_x(w, [b], np.arange(P))[0]
            dyb = ki.prefill_dy(w, [b], np.arange(P))[0]
            dx, gr = fn(xb, wts, w.tau, w.a, w.g, w.d_h, w.rope_base, dyb)
            dxs.append(dx)
            if tot is None:
                tot = gr
            else:
                for l in range(w.L):
                    for k, v in gr[l].items():
                        if v is not None:
                            tot[l][k] = tot[l][k] + v
        out.append((dxs, tot))
    return out
