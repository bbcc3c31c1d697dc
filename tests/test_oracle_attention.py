"""Pins for the attention oracle: a library routine (torch SDPA in fp64 on the
CPU), closed forms, invariants of Eqs. (1)-(3), brute force on tiny inputs,
and prefill/decode consistency."""
import math

import numpy as np
import pytest
import torch

from oracle import attention as at


def rng(seed=0):
    return np.random.default_rng(seed)


def sdpa(q, k, v, r):
    """torch's fp64 causal attention with the KV heads repeated r times."""
    qt = torch.from_numpy(q)[None]
    kt = torch.from_numpy(np.repeat(k, r, axis=0))[None]
    vt = torch.from_numpy(np.repeat(v, r, axis=0))[None]
    return torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, is_causal=True)[0].numpy()


@pytest.mark.parametrize("a,g,S,d", [(4, 4, 37, 16), (8, 2, 64, 32), (6, 3, 5, 8)])
def test_attention_matches_library_causal_sdpa(a, g, S, d):
    r = rng(a * 100 + S)
    q, k, v = r.normal(size=(a, S, d)), r.normal(size=(g, S, d)), r.normal(size=(g, S, d))
    out = at.attention(q, k, v, np.arange(S), np.arange(S))
    np.testing.assert_allclose(out, sdpa(q, k, v, a // g), rtol=1e-12, atol=1e-12)


def test_softmax_rows_sum_to_one_and_mask():
    r = rng(1)
    q, k, v = r.normal(size=(2, 20, 8)), r.normal(size=(1, 20, 8)), r.normal(size=(1, 20, 8))
    _, probs = at.attention(q, k, v, np.arange(20), np.arange(20), return_probs=True)
    for p in probs:
        np.testing.assert_allclose(p.sum(axis=1), 1.0, rtol=0, atol=1e-14)
        assert np.all(p[np.triu_indices(20, 1)] == 0.0)


def test_first_query_returns_first_value_and_equal_keys_average():
    r = rng(2)
    S, d = 12, 8
    q, v = r.normal(size=(4, S, d)), r.normal(size=(2, S, d))
    k = r.normal(size=(2, S, d))
    out = at.attention(q, k, v, np.arange(S), np.arange(S))
    # Position 0 sees only key 0: O = V[0] exactly.
    assert np.array_equal(out[:, 0], v[np.arange(4) // 2, 0])
    # All keys equal: uniform weights over the visible prefix -> running mean of V.
    k_eq = np.broadcast_to(r.normal(size=(1, 1, d)), (2, S, d)).copy()
    out = at.attention(q, k_eq, v, np.arange(S), np.arange(S))
    cm = np.cumsum(v, axis=1) / np.arange(1, S + 1)[None, :, None]
    np.testing.assert_allclose(out, cm[np.arange(4) // 2], rtol=1e-12, atol=1e-12)


def test_gqa_head_mapping_consecutive_groups():
    # Distinct constant V per kv head and equal keys: head j must return V of kv head j // r.
    a, g, S, d = 8, 2, 6, 4
    q = rng(3).normal(size=(a, S, d))
    k = np.zeros((g, S, d))
    v = np.stack([np.full((S, d), 10.0 * (kv + 1)) for kv in range(g)])
    out = at.attention(q, k, v, np.arange(S), np.arange(S))
    for j in range(a):
        np.testing.assert_allclose(out[j], 10.0 * (j // (a // g) + 1), rtol=1e-14)


def test_rope_closed_form_rotate_half():
    # e_i at position p -> cos(p theta_i) e_i + sin(p theta_i) e_{i + d/2}, theta_i = base^(-2i/d).
    d, base = 8, 10000.0
    for i in range(d // 2):
        x = np.zeros((1, d))
        x[0, i] = 1.0
        for p in (0, 1, 7, 1000):
            y = at.apply_rope(x, [p], base)[0]
            th = base ** (-2.0 * i / d)
            exp = np.zeros(d)
            exp[i] = math.cos(p * th)
            exp[i + d // 2] = math.sin(p * th)
            np.testing.assert_allclose(y, exp, atol=1e-15)
    # The partner of the upper half rotates the other way: e_{i+d/2} -> -sin e_i + cos e_{i+d/2}.
    x = np.zeros((1, d))
    x[0, d // 2] = 1.0
    y = at.apply_rope(x, [3], base)[0]
    assert abs(y[0] + math.sin(3.0)) < 1e-15 and abs(y[d // 2] - math.cos(3.0)) < 1e-15


def test_rope_norm_and_relative_position():
    r = rng(4)
    d = 64
    x = r.normal(size=(10, d))
    y = at.apply_rope(x, np.arange(10) * 37, 10000.0)
    np.testing.assert_allclose(np.linalg.norm(y, axis=1), np.linalg.norm(x, axis=1), rtol=1e-13)
    q, k = r.normal(size=(1, d)), r.normal(size=(1, d))
    dots = []
    for m, n in [(5, 2), (105, 102), (1003, 1000)]:
        dots.append((at.apply_rope(q, [m], 1e4) @ at.apply_rope(k, [n], 1e4).T).item())
    np.testing.assert_allclose(dots, dots[0], rtol=1e-10)


def _tiny_weights(r, L, h, a, g, d, tau, sigma=0.3):
    ws = []
    for l in range(L):
        prod = tau[l] == l
        ws.append(at.LayerWeights(r.normal(size=(a * d, h)) * sigma,
                                  r.normal(size=(g * d, h)) * sigma if prod else None,
                                  r.normal(size=(g * d, h)) * sigma if prod else None,
                                  r.normal(size=(h, a * d)) * sigma))
    return ws


def _brute_layer(x, w, a, g, d, base, kv=None):
    """Scalar loops straight from Eqs. (1)-(3), no vectorised helpers."""
    S, h = x.shape
    r = a // g

    def proj(W, n_out):
        return [[sum(x[s][c] * W[o][c] for c in range(h)) for o in range(n_out)] for s in range(S)]

    def rope(vec, p):
        half = d // 2
        out = [0.0] * d
        for i in range(half):
            th = p * base ** (-2.0 * i / d)
            out[i] = vec[i] * math.cos(th) - vec[i + half] * math.sin(th)
            out[i + half] = vec[i + half] * math.cos(th) + vec[i] * math.sin(th)
        return out

    Q = proj(w.wq, a * d)
    if kv is None:
        Kp, Vp = proj(w.wk, g * d), proj(w.wv, g * d)
        K = [[rope(Kp[s][kh * d:(kh + 1) * d], s) for s in range(S)] for kh in range(g)]
        V = [[Vp[s][kh * d:(kh + 1) * d] for s in range(S)] for kh in range(g)]
    else:
        K, V = kv
    O = [[0.0] * (a * d) for _ in range(S)]
    for j in range(a):
        kh = j // r
        for s in range(S):
            qv = rope(Q[s][j * d:(j + 1) * d], s)
            sc = [sum(qv[c] * K[kh][t][c] for c in range(d)) / math.sqrt(d) for t in range(s + 1)]
            mx = max(sc)
            e = [math.exp(v - mx) for v in sc]
            z = sum(e)
            for c in range(d):
                O[s][j * d + c] = sum(e[t] / z * V[kh][t][c] for t in range(s + 1))
    Y = [[x[s][c] + sum(O[s][m] * w.wo[c][m] for m in range(a * d)) for c in range(h)]
         for s in range(S)]
    return np.array(Y), np.array(O), (K, V)


def test_stack_matches_brute_force_loops():
    r = rng(5)
    L, h, a, g, d, S, base = 3, 8, 4, 2, 4, 6, 100.0
    tau = [0, 0, 2]
    ws = _tiny_weights(r, L, h, a, g, d, tau)
    x = r.normal(size=(S, h))
    y, xs, outs, caches = at.stack_prefill(x, ws, tau, a, g, d, base)
    cur = x
    kv0 = None
    for l in range(L):
        if tau[l] == l:
            cur_next, o, kv = _brute_layer(cur, ws[l], a, g, d, base)
            kv0 = kv
        else:
            cur_next, o, _ = _brute_layer(cur, ws[l], a, g, d, base, kv=kv0)
        np.testing.assert_allclose(outs[l], o, rtol=1e-11, atol=1e-12)
        cur = cur_next
    np.testing.assert_allclose(y, cur, rtol=1e-11, atol=1e-12)


def test_identity_map_is_standard_attention():
    r = rng(6)
    L, h, a, g, d, S = 2, 32, 4, 2, 8, 24
    tau = [0, 1]
    ws = _tiny_weights(r, L, h, a, g, d, tau)
    x = r.normal(size=(S, h))
    _, xs, outs, caches = at.stack_prefill(x, ws, tau, a, g, d, 10000.0)
    for l in range(L):
        q = at.apply_rope((xs[l] @ ws[l].wq.T).reshape(S, a, d).transpose(1, 0, 2), np.arange(S), 1e4)
        k, v = caches[l]
        ref = sdpa(q, k, v, a // g).transpose(1, 0, 2).reshape(S, a * d)
        np.testing.assert_allclose(outs[l], ref, rtol=1e-11, atol=1e-12)


def test_consumer_is_attention_on_producer_kv():
    r = rng(7)
    h, a, g, d, S = 32, 4, 2, 8, 24
    tau = [0, 0, 0]
    ws = _tiny_weights(r, 3, h, a, g, d, tau)
    x = r.normal(size=(S, h))
    _, xs, outs, caches = at.stack_prefill(x, ws, tau, a, g, d, 10000.0)
    assert list(caches) == [0]
    k0, v0 = caches[0]
    for l in (1, 2):
        q = at.apply_rope((xs[l] @ ws[l].wq.T).reshape(S, a, d).transpose(1, 0, 2), np.arange(S), 1e4)
        ref = sdpa(q, k0, v0, a // g).transpose(1, 0, 2).reshape(S, a * d)
        np.testing.assert_allclose(outs[l], ref, rtol=1e-11, atol=1e-12)
    # Sharing changes the result: giving layer 1 its own K/V does not reproduce it.
    ws_u = list(ws)
    ws_u[1] = at.LayerWeights(ws[1].wq, r.normal(size=(g * d, h)) * 0.3,
                              r.normal(size=(g * d, h)) * 0.3, ws[1].wo)
    _, _, outs_u, _ = at.stack_prefill(x, ws_u, [0, 1, 1], a, g, d, 10000.0)
    assert np.abs(outs_u[1] - outs[1]).max() > 1e-3


def test_decode_matches_prefill_row():
    """Decode at position p after a p-token prefill equals prefill row p."""
    r = rng(8)
    L, h, a, g, d, S = 4, 32, 4, 2, 8, 17
    tau = [0, 0, 2, 2]
    ws = _tiny_weights(r, L, h, a, g, d, tau)
    xs_full = r.normal(size=(S, h))
    y_full, xs, outs, caches_full = at.stack_prefill(xs_full, ws, tau, a, g, d, 10000.0)
    p = S - 1
    _, _, _, caches_p = at.stack_prefill(xs_full[:p], ws, tau, a, g, d, 10000.0)
    # Decode feeds the layer-0 input of row p; later layers see decode's own activations.
    y, outs_dec, new_kv = at.decode_step(xs_full[p], p, ws, tau, caches_p, a, g, d, 10000.0)
    np.testing.assert_allclose(y, y_full[p], rtol=1e-11, atol=1e-12)
    for l in range(L):
        np.testing.assert_allclose(outs_dec[l], outs[l][p], rtol=1e-11, atol=1e-12)
    for prod, (kn, vn) in new_kv.items():
        np.testing.assert_allclose(kn, caches_full[prod][0][:, p], rtol=1e-12, atol=1e-13)
        np.testing.assert_allclose(vn, caches_full[prod][1][:, p], rtol=1e-12, atol=1e-13)


def test_selected_rows_match_brute_force_and_causal_prefix():
    """layer_prefill on chosen query rows (producer and consumer) equals the brute-force
    scalar loops at those rows; a causal prefix of the input gives the same rows."""
    r = rng(9)
    h, a, g, d, S, base = 8, 4, 2, 4, 11, 100.0
    ws = _tiny_weights(r, 2, h, a, g, d, [0, 0])
    x = r.normal(size=(S, h))
    rows = [0, 3, 7, 10]
    y_b, o_b, kv_b = _brute_layer(x, ws[0], a, g, d, base)
    y, o, (k, v) = at.layer_prefill(x, ws[0], a, g, d, base, rows=rows)
    np.testing.assert_allclose(y, y_b[rows], rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(o, o_b[rows], rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(k, np.array(kv_b[0]), rtol=1e-11, atol=1e-12)
    x1 = r.normal(size=(S, h))
    y1_b, o1_b, _ = _brute_layer(x1, ws[1], a, g, d, base, kv=kv_b)
    y1, o1, _ = at.layer_prefill(x1, ws[1], a, g, d, base, shared_kv=(k, v), rows=rows)
    np.testing.assert_allclose(o1, o1_b[rows], rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(y1, y1_b[rows], rtol=1e-11, atol=1e-12)
    # Rows below n depend only on the first n inputs (the causal mask).
    n = 8
    yp, op, _ = at.layer_prefill(x[:n], ws[0], a, g, d, base, rows=[0, 3, 7])
    np.testing.assert_allclose(op, o_b[[0, 3, 7]], rtol=1e-11, atol=1e-12)
