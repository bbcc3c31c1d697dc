"""Oracle for the backward pass of the KV-shared attention stack (test
infrastructure only).

Plain fp64 NumPy, one sequence at a time, written from the chain rule on the
forward of ``oracle.attention`` (Sec. 2.2, Eqs. 1-3):

  Q_l = RoPE(X_l W_Q^T),  K_p = RoPE(X_p W_K^T),  V_p = X_p W_V^T  (producers p)
  O_l = softmax(Q_l K_tau(l)^T / sqrt(d_h) + M) V_tau(l)
  X_{l+1} = X_l + O_l W_O^T

Given dY = dLoss/dX_L it returns dLoss/dX_0 and the gradients of every
weight.  A consumer has no W_K, W_V (Eq. 3 drops them); the gradient that
reaches its producer's K and V through its attention adds to the producer's
own, so a producer's dW_K, dW_V and its dX carry the sum over the producer
and all of its consumers.  Training with KV sharing, as in Sec. 3, needs
exactly these gradients.
"""
from __future__ import annotations

import math
from typing import Dict, List, Sequence, Tuple

import numpy as np

from .attention import LayerWeights, _heads, _merge, apply_rope, attention, rope_cos_sin


def apply_rope_transpose(x: np.ndarray, positions: Sequence[int], base: float) -> np.ndarray:
    """The transpose of the RoPE rotation: rotate each pair (x_i, x_{i+d/2}) by -pos * theta_i.

    RoPE is linear and orthogonal per position, so the gradient with respect
    to its input is the gradient with respect to its output rotated back.
    """
    d_h = x.shape[-1]
    half = d_h // 2
    c, s = rope_cos_sin(positions, d_h, base)
    x1 = x[..., :half]
    x2 = x[..., half:]
    return np.concatenate([x1 * c + x2 * s, x2 * c - x1 * s], axis=-1)


def attention_backward(q: np.ndarray, k: np.ndarray, v: np.ndarray, do: np.ndarray,
                       q_pos: Sequence[int], k_pos: Sequence[int]):
    """Gradients of Eq. (2) for one sequence with GQA.

    q [a, Sq, d], k, v [g, Sk, d], do [a, Sq, d] -> (dq, dk, dv).  With
    S = q k^T / sqrt(d) (masked), P = softmax_rows(S) and O = P v:
    dv = P^T dO, dP = dO v^T, dS = P * (dP - rowsum(P * dP)) (the softmax
    Jacobian), dq = dS k / sqrt(d), dk = dS^T q / sqrt(d).  The r query heads
    that read one KV head add their dk, dv.
    """
    a, Sq, d = q.shape
    g = k.shape[0]
    r = a // g
    hidden = np.asarray(k_pos)[None, :] > np.asarray(q_pos)[:, None]
    dq = np.zeros_like(q, dtype=np.float64)
    dk = np.zeros(k.shape, dtype=np.float64)
    dv = np.zeros(v.shape, dtype=np.float64)
    inv = 1.0 / math.sqrt(d)
    for j in range(a):
        kv = j // r
        s = (q[j] @ k[kv].T) * inv
        s = np.where(hidden, -np.inf, s)
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p = p / p.sum(axis=1, keepdims=True)
        dv[kv] += p.T @ do[j]
        dp = do[j] @ v[kv].T
        ds = p * (dp - (p * dp).sum(axis=1, keepdims=True))
        dq[j] = (ds @ k[kv]) * inv
        dk[kv] += (ds.T @ q[j]) * inv
    return dq, dk, dv


def stack_backward(x: np.ndarray, weights: Sequence[LayerWeights], tau: Sequence[int], a: int,
                   g: int, d_h: int, base: float, dy: np.ndarray):
    """Backward of ``oracle.attention.stack_prefill`` for one sequence x [S, h].

    Returns (dx [S, h], grads) with grads[l] a dict of dwq, dwo and, for a
    producer, dwk, dwv ([out, in] like the weights; None for a consumer's
    dwk, dwv).  tau must be canonical (every tau(l) a producer).
    """
    S = x.shape[0]
    pos = np.arange(S)
    L = len(weights)
    for l in range(L):
        if int(tau[int(tau[l])]) != int(tau[l]) or int(tau[l]) > l:
            raise ValueError("tau must map every layer to a prior producer")
    # Forward, keeping what the backward needs.
    xs, qs, os_ = [], [], []
    kv: Dict[int, Tuple[np.ndarray, np.ndarray]] = {}
    cur = np.asarray(x, dtype=np.float64)
    for l, w in enumerate(weights):
        xs.append(cur)
        q = apply_rope(_heads(cur @ w.wq.T, a, d_h), pos, base)
        if int(tau[l]) == l:
            kv[l] = (apply_rope(_heads(cur @ w.wk.T, g, d_h), pos, base), _heads(cur @ w.wv.T, g, d_h))
        k, v = kv[int(tau[l])]
        o = _merge(attention(q, k, v, pos, pos))
        qs.append(q)
        os_.append(o)
        cur = cur + o @ w.wo.T
    # Backward, last layer first: every consumer of p (index > p) is done before p.
    grads: List[dict] = [None] * L
    dk_acc: Dict[int, np.ndarray] = {}
    dv_acc: Dict[int, np.ndarray] = {}
    gx = np.asarray(dy, dtype=np.float64)            # dLoss / dX_{l+1}
    for l in range(L - 1, -1, -1):
        w = weights[l]
        p = int(tau[l])
        dwo = gx.T @ os_[l]
        do = _heads(gx @ w.wo, a, d_h)
        k, v = kv[p]
        dq, dk, dv = attention_backward(qs[l], k, v, do, pos, pos)
        dk_acc[p] = dk_acc.get(p, 0.0) + dk
        dv_acc[p] = dv_acc.get(p, 0.0) + dv
        dq_pre = _merge(apply_rope_transpose(dq, pos, base))          # [S, a d]
        gnew = gx + dq_pre @ w.wq
        gr = {"dwq": dq_pre.T @ xs[l], "dwo": dwo, "dwk": None, "dwv": None}
        if p == l:
            dk_pre = _merge(apply_rope_transpose(dk_acc.pop(l), pos, base))   # [S, g d]
            dv_all = _merge(dv_acc.pop(l))
            gr["dwk"] = dk_pre.T @ xs[l]
            gr["dwv"] = dv_all.T @ xs[l]
            gnew = gnew + dk_pre @ w.wk + dv_all @ w.wv
        grads[l] = gr
        gx = gnew
    return gx, grads

