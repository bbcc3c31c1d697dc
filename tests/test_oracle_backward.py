"""Pins for the backward oracle: central finite differences of the forward
oracle, torch fp64 autograd through an independent torch forward (library
routines), closed forms of the softmax Jacobian, and RoPE orthogonality."""
import math

import numpy as np
import pytest
import torch

from oracle import attention as at
from oracle import backward as bw


def make_stack(seed, L, h, a, g, d, tau, wscale=0.3):
    r = np.random.default_rng(seed)
    ws = []
    for l in range(L):
        prod = tau[l] == l
        ws.append(at.LayerWeights(r.normal(size=(a * d, h)) * wscale,
                                  r.normal(size=(g * d, h)) * wscale if prod else None,
                                  r.normal(size=(g * d, h)) * wscale if prod else None,
                                  r.normal(size=(h, a * d)) * wscale))
    return ws


def loss(x, ws, tau, a, g, d, base, dy):
    y = at.stack_prefill(x, ws, tau, a, g, d, base)[0]
    return float(np.sum(y * dy))


CASES = [
    # L, h, a, g, d, S, tau, base
    (3, 8, 2, 2, 4, 5, [0, 0, 2], 10.0),          # MHA, one consumer
    (4, 12, 4, 2, 3 * 2, 6, [0, 0, 0, 3], 100.0),  # GQA r = 2, two consumers of layer 0
    (2, 8, 4, 1, 2 * 2, 4, [0, 1], 10000.0),     # MQA r = 4, identity map
]


@pytest.mark.parametrize("L,h,a,g,d,S,tau,base", CASES)
def test_directional_finite_differences(L, h, a, g, d, S, tau, base):
    r = np.random.default_rng(L * 10 + h)
    ws = make_stack(L + h, L, h, a, g, d, tau)
    x = r.normal(size=(S, h))
    dy = r.normal(size=(S, h))
    dx, grads = bw.stack_backward(x, ws, tau, a, g, d, base, dy)
    eps = 1e-4

    def check(analytic, perturb):
        # Five-point central difference, truncation error O(eps^4).
        u = r.normal(size=analytic.shape)
        f = {m: loss(*perturb(u, m * eps), tau, a, g, d, base, dy) for m in (-2, -1, 1, 2)}
        fd = (f[-2] - 8 * f[-1] + 8 * f[1] - f[2]) / (12 * eps)
        an = float(np.sum(analytic * u))
        assert abs(fd - an) <= 1e-8 * max(1.0, abs(an)), (fd, an)

    check(dx, lambda u, e: (x + e * u, ws))
    for l in range(L):
        for name in ("wq", "wk", "wv", "wo"):
            gval = grads[l]["d" + name]
            if getattr(ws[l], name) is None:
                assert gval is None
                continue

            def pert(u, e, l=l, name=name):
                ws2 = [at.LayerWeights(w.wq, w.wk, w.wv, w.wo) for w in ws]
                setattr(ws2[l], name, getattr(ws[l], name) + e * u)
                return x, ws2
            check(gval, pert)


def torch_forward(x, ws, tau, a, g, d, base):
    """The stack in torch fp64 ops with SDPA; autograd supplies the backward."""
    S = x.shape[0]
    half = d // 2
    theta = base ** (-2.0 * torch.arange(half, dtype=torch.float64) / d)
    ang = torch.arange(S, dtype=torch.float64)[:, None] * theta[None, :]
    c, s = torch.cos(ang), torch.sin(ang)

    def rope(t):        # t [n, S, d]
        t1, t2 = t[..., :half], t[..., half:]
        return torch.cat([t1 * c - t2 * s, t2 * c + t1 * s], dim=-1)

    cache = {}
    cur = x
    for l, w in enumerate(ws):
        q = rope((cur @ w["wq"].T).reshape(S, a, d).transpose(0, 1))
        if tau[l] == l:
            k = rope((cur @ w["wk"].T).reshape(S, g, d).transpose(0, 1))
            v = (cur @ w["wv"].T).reshape(S, g, d).transpose(0, 1)
            cache[l] = (k, v)
        k, v = cache[tau[l]]
        o = torch.nn.functional.scaled_dot_product_attention(
            q[None], k.repeat_interleave(a // g, dim=0)[None].contiguous(),
            v.repeat_interleave(a // g, dim=0)[None].contiguous(), is_causal=True)[0]
        cur = cur + o.transpose(0, 1).reshape(S, a * d) @ w["wo"].T
    return cur


@pytest.mark.parametrize("L,h,a,g,d,S,tau,base", CASES + [(5, 16, 8, 2, 4, 17, [0, 0, 2, 2, 2], 10000.0)])
def test_matches_torch_autograd(L, h, a, g, d, S, tau, base):
    r = np.random.default_rng(7 + L)
    ws = make_stack(3 * L, L, h, a, g, d, tau)
    x = r.normal(size=(S, h))
    dy = r.normal(size=(S, h))
    dx, grads = bw.stack_backward(x, ws, tau, a, g, d, base, dy)
    xt = torch.tensor(x, requires_grad=True)
    wt = [{n: (torch.tensor(getattr(w, n), requires_grad=True) if getattr(w, n) is not None else None)
           for n in ("wq", "wk", "wv", "wo")} for w in ws]
    y = torch_forward(xt, wt, tau, a, g, d, base)
    (y * torch.from_numpy(dy)).sum().backward()
    np.testing.assert_allclose(dx, xt.grad.numpy(), rtol=1e-10, atol=1e-10)
    for l in range(L):
        for n in ("wq", "wk", "wv", "wo"):
            if wt[l][n] is None:
                assert grads[l]["d" + n] is None
            else:
                np.testing.assert_allclose(grads[l]["d" + n], wt[l][n].grad.numpy(), rtol=1e-10, atol=1e-10)


def test_softmax_jacobian_closed_forms():
    r = np.random.default_rng(11)
    a, g, S, d = 4, 2, 9, 8
    q, v, do = r.normal(size=(a, S, d)), r.normal(size=(g, S, d)), r.normal(size=(a, S, d))
    k = r.normal(size=(g, S, d))
    pos = np.arange(S)
    dq, dk, dv = bw.attention_backward(q, k, v, do, pos, pos)
    # Query 0 sees one key: P = 1, so its score gradient and dq vanish.
    assert np.all(dq[:, 0] == 0.0)
    # Rows of dS sum to zero, hence sum over keys of dk is sum over queries of dS^T q = ... and,
    # with all keys equal, dq = k * rowsum(dS) / sqrt(d) = 0 and P is uniform over the prefix:
    # dv[key] = sum over q >= key of do[q] / (q + 1), summed over the r heads.
    k_eq = np.broadcast_to(r.normal(size=(g, 1, d)), (g, S, d)).copy()
    dq, dk, dv = bw.attention_backward(q, k_eq, v, do, pos, pos)
    np.testing.assert_allclose(dq, 0.0, atol=1e-12)
    w = do / (pos + 1.0)[None, :, None]
    tail = np.cumsum(w[:, ::-1], axis=1)[:, ::-1]              # sum over q >= key
    ref = tail.reshape(g, a // g, S, d).sum(axis=1)
    np.testing.assert_allclose(dv, ref, rtol=1e-12, atol=1e-12)
    # A zero upstream gradient gives zero everywhere.
    z = bw.attention_backward(q, k, v, np.zeros_like(do), pos, pos)
    assert all(np.all(t == 0) for t in z)


def test_rope_transpose_is_inverse_and_adjoint():
    r = np.random.default_rng(12)
    x, y = r.normal(size=(3, 10, 16)), r.normal(size=(3, 10, 16))
    pos = np.arange(10) * 7
    rx = at.apply_rope(x, pos, 10000.0)
    np.testing.assert_allclose(bw.apply_rope_transpose(rx, pos, 10000.0), x, rtol=1e-12, atol=1e-12)
    lhs = np.sum(rx * y)
    rhs = np.sum(x * bw.apply_rope_transpose(y, pos, 10000.0))
    assert abs(lhs - rhs) < 1e-10


def test_consumer_gradient_reaches_producer_weights():
    # With a consumer, the producer's dW_K is its own plus the consumer's contribution:
    # zeroing the consumer's W_O removes that contribution exactly.
    L, h, a, g, d, S = 2, 8, 2, 1, 4, 6
    r = np.random.default_rng(13)
    ws = make_stack(1, L, h, a, g, d, [0, 0])
    x, dy = r.normal(size=(S, h)), r.normal(size=(S, h))
    _, gr_shared = bw.stack_backward(x, ws, [0, 0], a, g, d, 10.0, dy)
    ws0 = [ws[0], at.LayerWeights(ws[1].wq, None, None, np.zeros_like(ws[1].wo))]
    _, gr_cut = bw.stack_backward(x, ws0, [0, 0], a, g, d, 10.0, dy)
    # The producer alone (one-layer stack) sees the same upstream gradient when layer 1 adds 0.
    _, gr_one = bw.stack_backward(x, [ws[0]], [0], a, g, d, 10.0, dy)
    np.testing.assert_allclose(gr_cut[0]["dwk"], gr_one[0]["dwk"], rtol=1e-12, atol=1e-12)
    assert np.abs(gr_shared[0]["dwk"] - gr_one[0]["dwk"]).max() > 1e-3
