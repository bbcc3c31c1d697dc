"""Oracle for the KV-shared attention stack (test infrastructure only).

Plain fp64 NumPy, one sequence at a time (rows of a batch never interact).

Sec. 2.2: a full-attention layer projects Q, K, V from its hidden states and
computes softmax(Q K^T / sqrt(d_h) + M) V with the causal mask M (Eqs. 1-2);
during decoding it appends its K, V to the cache.  A KV-sharing layer keeps
its own query projection and the attention formula but takes K and V from a
prior layer tau(l) (Eq. 3).

Readings where the paper is silent (each is pinned by a test):
* RoPE uses the rotate-half pairing (x_i, x_{i+d/2}) with
  theta_i = base^(-2i/d_h); it rotates Q of every layer and K of producers
  before K is cached, so a consumer reuses post-RoPE keys.
* Query head j reads KV head floor(j / r), r = a / g.
* The stack is attention-only with a residual: X_{l+1} = X_l + O_l W_O^T.
* Decode: the new token sits at position p = current length; a producer
  appends its K, V at p before attending, so every layer attends over p + 1
  keys.
"""
from __future__ import annotations

import math
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np


def rope_cos_sin(positions: Sequence[int], d_h: int, base: float) -> Tuple[np.ndarray, np.ndarray]:
    """cos/sin of pos * theta_i, theta_i = base^(-2i/d_h), i < d_h/2 -> two [n_pos, d_h/2] arrays."""
    half = d_h // 2
    i = np.arange(half, dtype=np.float64)
    theta = np.power(float(base), -2.0 * i / d_h)
    ang = np.asarray(positions, dtype=np.float64)[:, None] * theta[None, :]
    return np.cos(ang), np.sin(ang)


def apply_rope(x: np.ndarray, positions: Sequence[int], base: float) -> np.ndarray:
    """Rotate the pairs (x_i, x_{i+d/2}) of x[..., n_pos, d_h] by pos * theta_i."""
    d_h = x.shape[-1]
    half = d_h // 2
    c, s = rope_cos_sin(positions, d_h, base)
    x1 = x[..., :half]
    x2 = x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, q_pos: Sequence[int],
              k_pos: Sequence[int], return_probs: bool = False):
    """Eq. (2) for one sequence with GQA: q [a, Sq, d], k, v [g, Sk, d] -> [a, Sq, d].

    Key n is visible to query m iff k_pos[n] <= q_pos[m] (the causal mask M).
    """
    a, Sq, d = q.shape
    g = k.shape[0]
    if a % g:
        raise ValueError("query heads must be a multiple of kv heads")
    r = a // g
    qp = np.asarray(q_pos)[:, None]
    kp = np.asarray(k_pos)[None, :]
    hidden = kp > qp
    out = np.empty((a, Sq, v.shape[-1]), dtype=np.float64)
    probs = [] if return_probs else None
    for j in range(a):
        kv = j // r
        s = (q[j] @ k[kv].T) / math.sqrt(d)
        s = np.where(hidden, -np.inf, s)
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p = p / p.sum(axis=1, keepdims=True)
        out[j] = p @ v[kv]
        if return_probs:
            probs.append(p)
    return (out, probs) if return_probs else out


def _heads(x: np.ndarray, n: int, d: int) -> np.ndarray:
    """[S, n*d] -> [n, S, d]."""
    return x.reshape(x.shape[0], n, d).transpose(1, 0, 2)


def _merge(x: np.ndarray) -> np.ndarray:
    """[n, S, d] -> [S, n*d]."""
    n, S, d = x.shape
    return x.transpose(1, 0, 2).reshape(S, n * d)


class LayerWeights:
    """fp64 weights of one layer, [out, in] row-major; wk/wv are None for consumers."""

    def __init__(self, wq, wk, wv, wo):
        self.wq = np.asarray(wq, dtype=np.float64)
        self.wk = None if wk is None else np.asarray(wk, dtype=np.float64)
        self.wv = None if wv is None else np.asarray(wv, dtype=np.float64)
        self.wo = np.asarray(wo, dtype=np.float64)


def project_qkv(x: np.ndarray, positions: Sequence[int], w: LayerWeights, a: int, g: int, d_h: int,
                base: float, kv: bool = True):
    """Eq. (1) for the rows x [n, h] at the given absolute positions, with RoPE on Q and K.

    Returns (q [a, n, d_h], k [g, n, d_h] or None, v [g, n, d_h] or None); K and V are
    computed only when ``kv`` is set (a producer).
    """
    q = apply_rope(_heads(x @ w.wq.T, a, d_h), positions, base)
    if not kv:
        return q, None, None
    k = apply_rope(_heads(x @ w.wk.T, g, d_h), positions, base)
    v = _heads(x @ w.wv.T, g, d_h)
    return q, k, v


def output_projection(x: np.ndarray, o: np.ndarray, w: LayerWeights) -> np.ndarray:
    """The residual block output X + O W_O^T for rows x [n, h] and attention outputs o [n, a*d_h]."""
    return x + o @ w.wo.T


def layer_prefill(x: np.ndarray, w: LayerWeights, a: int, g: int, d_h: int, base: float,
                  shared_kv: Optional[Tuple[np.ndarray, np.ndarray]] = None,
                  rows: Optional[Sequence[int]] = None):
    """One layer over one sequence x [S, h].

    Producer (shared_kv is None): Q, K, V from x (Eq. 1), RoPE on Q and K.
    Consumer: Q from x, K and V = the producer's post-RoPE K, V (Eq. 3).
    ``rows`` (default: all S positions) selects the query positions whose outputs are
    computed; a producer still projects K and V at every position of x.
    Returns (x_next [n, h], o [n, a*d_h], (K, V) used, each [g, S, d_h]) for the n
    selected rows.
    """
    S = x.shape[0]
    pos = np.arange(S)
    qpos = pos if rows is None else np.asarray(rows)
    q, _, _ = project_qkv(x[qpos], qpos, w, a, g, d_h, base, kv=False)
    if shared_kv is None:
        _, k, v = project_qkv(x, pos, w, a, g, d_h, base)
    else:
        k, v = shared_kv
    o = _merge(attention(q, k, v, qpos, np.arange(k.shape[1])))
    return output_projection(x[qpos], o, w), o, (k, v)


def stack_prefill(x: np.ndarray, weights: Sequence[LayerWeights], tau: Sequence[int], a: int,
                  g: int, d_h: int, base: float):
    """Run every layer in order for one sequence.

    Returns (final x [S, h], per-layer inputs, per-layer attention outputs,
    dict producer -> (K, V) post-RoPE caches).
    """
    caches: Dict[int, Tuple[np.ndarray, np.ndarray]] = {}
    xs, outs = [], []
    cur = np.asarray(x, dtype=np.float64)
    for l, wl in enumerate(weights):
        p = int(tau[l])
        xs.append(cur)
        if p == l:
            cur, o, kv = layer_prefill(cur, wl, a, g, d_h, base)
            caches[l] = kv
        else:
            cur, o, _ = layer_prefill(cur, wl, a, g, d_h, base, shared_kv=caches[p])
        outs.append(o)
    return cur, xs, outs, caches


def decode_step(x: np.ndarray, pos: int, weights: Sequence[LayerWeights], tau: Sequence[int],
                caches: Dict[int, Tuple[np.ndarray, np.ndarray]], a: int, g: int, d_h: int,
                base: float):
    """One new token of one sequence at position ``pos`` through the stack.

    ``caches[p]`` holds the producer's post-RoPE K, V for positions [0, pos)
    as [g, >= pos, d_h]; only the first ``pos`` positions are read.
    Returns (y [h], per-layer attention outputs [a*d_h], dict producer ->
    (k_new, v_new) [g, d_h] appended at ``pos``).
    """
    cur = np.asarray(x, dtype=np.float64)[None, :]
    outs = []
    new_kv: Dict[int, Tuple[np.ndarray, np.ndarray]] = {}
    full: Dict[int, Tuple[np.ndarray, np.ndarray]] = {}
    for l, wl in enumerate(weights):
        p = int(tau[l])
        q = apply_rope(_heads(cur @ wl.wq.T, a, d_h), [pos], base)
        if p == l:
            k_new = apply_rope(_heads(cur @ wl.wk.T, g, d_h), [pos], base)
            v_new = _heads(cur @ wl.wv.T, g, d_h)
            kc, vc = caches[l]
            full[l] = (np.concatenate([np.asarray(kc[:, :pos], np.float64), k_new], axis=1),
                       np.concatenate([np.asarray(vc[:, :pos], np.float64), v_new], axis=1))
            new_kv[l] = (k_new[:, 0, :], v_new[:, 0, :])
        k, v = full[p]
        o = _merge(attention(q, k, v, [pos], np.arange(pos + 1)))
        outs.append(o[0])
        cur = cur + o @ wl.wo.T
    return cur[0], outs, new_kv
