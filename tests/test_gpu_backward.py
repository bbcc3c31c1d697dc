"""GPU parity of the training path through the C ABI: kvp_train_forward (same output
as kvp_prefill, plus saved activations) and kvp_backward against the fp64 backward
oracle, on the same seeded inputs: dX and every weight gradient, with producers
that have zero, one and two consumers, GQA ratios 1, 2 and 4, ragged S and S = 1; bf16
models at 2e-2 of max|ref| per tensor, fp32 models (the tiny fp32 configuration among
them) at 1e-5."""
import numpy as np
import pytest
import torch

import kvp_inputs as ki
from kvp_inputs import device as kd
from oracle import backward as obw
from paper_2608_15943_amd import binding as kb

from gpu_util import (DEV, build_device_model, oracle_weights, rel_err, say, small_workload, tdtype,
                      to_np, workspace)
from gpu_util import tol as tol_for

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    kb.lib()


TOL = 2e-2   # bf16 path: max|err| <= 2e-2 max|ref| per tensor


def _train_case(w, B, S, cap):
    say(f"[backward] {w.name} {w.dtype} B={B} S={S} tau={w.tau}")
    tol = tol_for(w)
    dm = build_device_model(w, B, S, cap)
    m = dm.model
    st = torch.cuda.current_stream().cuda_stream
    x = torch.empty((B, S, w.h), dtype=tdtype(w), device=DEV)
    kd.fill_prefill_x(w, x.data_ptr(), B, S)
    y = torch.empty_like(x)
    y_ref = torch.empty_like(x)
    ws, n = workspace(dm, kb.KVP_PHASE_PREFILL, B, S)
    m.kvp_prefill(x.data_ptr(), y_ref.data_ptr(), B, S, ws.data_ptr(), n, st)
    nsv = m.kvp_train_saved_size(B, S)
    saved = torch.empty(nsv, dtype=torch.uint8, device=DEV)
    m.kvp_train_forward(x.data_ptr(), y.data_ptr(), B, S, saved.data_ptr(), nsv, ws.data_ptr(), n, st)
    torch.cuda.synchronize()
    # The training forward runs the same kernels: same output bit for bit.
    assert torch.equal(y, y_ref)

    grads = {}
    for l in range(w.L):
        prod = w.tau[l] == l
        gq = torch.full((w.a * w.d_h, w.h), float("nan"), device=DEV)
        go = torch.full((w.h, w.a * w.d_h), float("nan"), device=DEV)
        gk = torch.full((w.g * w.d_h, w.h), float("nan"), device=DEV) if prod else None
        gv = torch.full((w.g * w.d_h, w.h), float("nan"), device=DEV) if prod else None
        m.kvp_set_layer_grads(l, gq.data_ptr(), gk.data_ptr() if prod else 0,
                              gv.data_ptr() if prod else 0, go.data_ptr())
        grads[l] = {"dwq": gq, "dwk": gk, "dwv": gv, "dwo": go}
    dy = torch.empty((B, S, w.h), dtype=torch.float32, device=DEV)
    kd.fill_prefill_dy(w, dy.data_ptr(), B, S)
    dx = torch.full_like(dy, float("nan"))
    wsb, nb = workspace(dm, kb.KVP_PHASE_BACKWARD, B, S)
    m.kvp_backward(x.data_ptr(), dy.data_ptr(), dx.data_ptr(), B, S, saved.data_ptr(), nsv,
                   wsb.data_ptr(), nb, st)
    torch.cuda.synchronize()
    say("  backward done; oracle ...")

    wts = oracle_weights(w)
    ref_g = None
    worst = 0.0
    for b in range(B):
        xb = ki.prefill_x(w, [b], np.arange(S))[0]
        dyb = ki.prefill_dy(w, [b], np.arange(S))[0]
        dxb, gb = obw.stack_backward(xb, wts, w.tau, w.a, w.g, w.d_h, w.rope_base, dyb)
        e = rel_err(to_np(dx[b]), dxb)
        say(f"  dx[{b}]: {e:.3e}")
        worst = max(worst, e)
        assert e <= tol, ("dx", b, e)
        if ref_g is None:
            ref_g = gb
        else:
            for l in range(w.L):
                for k, v in gb[l].items():
                    if v is not None:
                        ref_g[l][k] = ref_g[l][k] + v
    for l in range(w.L):
        p = w.tau[l]
        for k in ("dwq", "dwk", "dwv", "dwo"):
            if ref_g[l][k] is None:
                assert grads[l][k] is None
                continue
            got = to_np(grads[l][k])
            if S == 1 and k in ("dwq", "dwk"):
                # One visible key: the softmax Jacobian is zero, so dQ = dK = 0 exactly;
                # the kernels may leave a rounding residual of dP - D, bounded here by the
                # tolerance against the same attention's value-path gradient dW_V.
                assert np.abs(ref_g[l][k]).max() < 1e-12
                scale = np.abs(ref_g[p]["dwv"]).max()
                e = float(np.abs(got).max() / scale)
            else:
                e = rel_err(got, ref_g[l][k])
            say(f"  layer {l} {k}: {e:.3e}")
            worst = max(worst, e)
            assert e <= tol, (l, k, e)
    say(f"  max rel err {worst:.3e}")


@pytest.mark.parametrize("h,a,g,tau,B,S", [
    (256, 2, 1, [0, 0, 2], 2, 200),          # r = 2, one consumer, ragged S over two key blocks
    (512, 4, 2, [0, 0, 0, 3], 1, 300),       # two consumers add into one producer
    (256, 2, 2, [0, 1], 1, 64),              # MHA, identity map, one tile
    (512, 4, 1, [0, 1, 1], 3, 130),          # r = 4, batch of 3, S just past a key block
    (256, 2, 1, [0, 0], 2, 1),               # S = 1
    (256, 2, 1, [0, 0, 2], 2, 256),          # 512 tokens: weight gradients on token-major copies
    (1024, 8, 1, [0, 0], 1, 160),            # r = 8 (the 70B-shaped ratio), one consumer
    # Token counts that are multiples of 512 with S % 8 == 0: the attention kernels write O^T
    # and [dQ|dK|dV]^T themselves; S below a 32-token wave block (8), and one full block plus
    # an 8-token tail (40), take the partial-run stores.
    (256, 2, 1, [0, 0], 64, 8),
    (256, 2, 1, [0, 0, 2], 64, 40),
])
def test_backward_matches_oracle(h, a, g, tau, B, S):
    w = small_workload(f"bwd-h{h}-a{a}-g{g}", len(tau), h, a, g, tau, seed=21)
    cap = (S + 63) // 64 * 64
    _train_case(w, B, S, cap)


def test_backward_tiny_fp32_config():
    """The tiny fp32 configuration (4 layers, d_model 256, 4 x 64 heads, S 128, map
    [0, 0, 2, 2]) through the fp32 training path, at 1e-5."""
    w = ki.tiny_fp32()
    _train_case(w, w.batch, w.seq, w.kv_capacity)


@pytest.mark.parametrize("h,a,g,d,tau,B,S", [
    (128, 4, 2, 32, [0, 0, 2], 2, 37),       # GQA r = 2, ragged S, one consumer
    (64, 4, 1, 16, [0, 0, 0], 1, 50),        # r = 4, two consumers of one producer
    (128, 2, 2, 64, [0, 0], 2, 1),           # S = 1
])
def test_backward_fp32_matches_oracle(h, a, g, d, tau, B, S):
    w = small_workload(f"bwd32-h{h}-a{a}-g{g}-d{d}", len(tau), h, a, g, tau, dtype="fp32", d_h=d, seed=23)
    _train_case(w, B, S, S + 3)



def _prefix_case(w, B, S, P, tol_dx, tol_w):
    """Training step of workload w at (B, S) with dY zero past position P: the loss reads only
    outputs at positions < P, which depend only on inputs before P (causal stack), so every
    gradient equals that of the P-token problem, which the oracle solves for all sequences;
    dX past P is exactly 0."""
    say(f"[backward full] {w.name} L={w.L} B={B} S={S} tau={w.tau}, dY zero past {P}")
    dm = build_device_model(w, B, S, w.kv_capacity)
    m = dm.model
    st = torch.cuda.current_stream().cuda_stream
    x = torch.empty((B, S, w.h), dtype=torch.bfloat16, device=DEV)
    kd.fill_prefill_x(w, x.data_ptr(), B, S)
    y = torch.empty_like(x)
    ws, n = workspace(dm, kb.KVP_PHASE_PREFILL, B, S)
    nsv = m.kvp_train_saved_size(B, S)
    saved = torch.empty(nsv, dtype=torch.uint8, device=DEV)
    m.kvp_train_forward(x.data_ptr(), y.data_ptr(), B, S, saved.data_ptr(), nsv, ws.data_ptr(), n, st)
    grads = {}
    for l in range(w.L):
        prod = w.tau[l] == l
        g = {"dwq": torch.empty((w.a * w.d_h, w.h), device=DEV), "dwo": torch.empty((w.h, w.a * w.d_h), device=DEV),
             "dwk": torch.empty((w.g * w.d_h, w.h), device=DEV) if prod else None,
             "dwv": torch.empty((w.g * w.d_h, w.h), device=DEV) if prod else None}
        m.kvp_set_layer_grads(l, g["dwq"].data_ptr(), g["dwk"].data_ptr() if prod else 0,
                              g["dwv"].data_ptr() if prod else 0, g["dwo"].data_ptr())
        grads[l] = g
    dy = torch.empty((B, S, w.h), dtype=torch.float32, device=DEV)
    kd.fill_prefill_dy(w, dy.data_ptr(), B, S)
    dy[:, P:] = 0
    dx = torch.empty_like(dy)
    wsb, nb = workspace(dm, kb.KVP_PHASE_BACKWARD, B, S)
    m.kvp_backward(x.data_ptr(), dy.data_ptr(), dx.data_ptr(), B, S, saved.data_ptr(), nsv,
                   wsb.data_ptr(), nb, st)
    torch.cuda.synchronize()
    assert bool((dx[:, P:] == 0).all().item()), "dX past the prefix must be zero"
    say("  backward done; oracle on the prefix ...")
    wts = oracle_weights(w)
    ref_g = None
    e_dx = 0.0
    for b in range(B):
        xb = ki.prefill_x(w, [b], np.arange(P))[0]
        dyb = ki.prefill_dy(w, [b], np.arange(P))[0]
        dxb, gb = obw.stack_backward(xb, wts, w.tau, w.a, w.g, w.d_h, w.rope_base, dyb)
        e = rel_err(to_np(dx[b, :P]), dxb)
        say(f"  dx[{b}]: {e:.3e}")
        e_dx = max(e_dx, e)
        if ref_g is None:
            ref_g = gb
        else:
            for l in range(w.L):
                for k, v in gb[l].items():
                    if v is not None:
                        ref_g[l][k] = ref_g[l][k] + v
    e_w = 0.0
    for l in range(w.L):
        for k in ("dwq", "dwk", "dwv", "dwo"):
            if ref_g[l][k] is not None:
                e = rel_err(to_np(grads[l][k]), ref_g[l][k])
                say(f"  layer {l} {k}: {e:.3e}")
                e_w = max(e_w, e)
    say(f"  max rel err: dx {e_dx:.3e}, weight gradients {e_w:.3e}")
    del dm, x, y, saved, ws, wsb, dy, dx, grads
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    assert e_dx <= tol_dx and e_w <= tol_w, (e_dx, e_w)


def test_backward_full_size_three_layers():
    """Three layers of the 8-layer stage's shape (d_model 2048, 16 / 8 heads) at its batch and
    length (B 4, S 4096), in the benchmark's launch configuration: a producer with no consumer
    and a producer with one, at the 2e-2 bar."""
    w = ki.Workload(name="stage-shape-3L", L=3, h=2048, a=16, g=8, d_h=128, dtype="bf16",
                    tau=[0, 1, 1], phase="prefill", batch=4, seq=4096, kv_capacity=4096, seed=5)
    _prefix_case(w, 4, 4096, 300, TOL, TOL)


def test_backward_stage_share_full_size_prefix():
    """The 8-layer stage share itself, composed.  Its gradients are bounded by what bf16
    forward activations allow: the precision model of tests/bf16_emulation.py (the oracle with
    the layer inputs, Q, K, V and O rounded to bf16, otherwise exact) moves this problem's dX
    by 2.8e-2 and its weight gradients by 3.5e-2 of max|ref| (test_bf16_backward_bound.py
    reproduces this on the CPU), so the bound here is 5e-2.  (The GPU is not closer to that
    model than to the exact oracle: the deep stack amplifies which way each rounding goes, so
    two bf16 realizations differ from each other by as much as from the exact result.)  The
    three-layer test above holds the 2e-2 bar."""
    w = ki.stage_share_prefill()
    _prefix_case(w, w.batch, w.seq, 300, 5e-2, 5e-2)


def _train_outputs(w, B, S, cap, fill):
    dm = build_device_model(w, B, S, cap)
    for K, V in dm.slots.values():
        K.fill_(fill)
        V.fill_(fill)
    m = dm.model
    st = torch.cuda.current_stream().cuda_stream
    x = torch.empty((B, S, w.h), dtype=torch.bfloat16, device=DEV)
    kd.fill_prefill_x(w, x.data_ptr(), B, S)
    y = torch.empty_like(x)
    ws, n = workspace(dm, kb.KVP_PHASE_PREFILL, B, S)
    nsv = m.kvp_train_saved_size(B, S)
    saved = torch.empty(nsv, dtype=torch.uint8, device=DEV)
    m.kvp_train_forward(x.data_ptr(), y.data_ptr(), B, S, saved.data_ptr(), nsv, ws.data_ptr(), n, st)
    outs = [y]
    for l in range(w.L):
        prod = w.tau[l] == l
        g = [torch.empty((w.a * w.d_h, w.h), device=DEV), torch.empty((w.g * w.d_h, w.h), device=DEV) if prod else None,
             torch.empty((w.g * w.d_h, w.h), device=DEV) if prod else None, torch.empty((w.h, w.a * w.d_h), device=DEV)]
        m.kvp_set_layer_grads(l, *[t.data_ptr() if t is not None else 0 for t in g])
        outs += [t for t in g if t is not None]
    dy = torch.empty((B, S, w.h), dtype=torch.float32, device=DEV)
    kd.fill_prefill_dy(w, dy.data_ptr(), B, S)
    dx = torch.empty_like(dy)
    wsb, nb = workspace(dm, kb.KVP_PHASE_BACKWARD, B, S)
    m.kvp_backward(x.data_ptr(), dy.data_ptr(), dx.data_ptr(), B, S, saved.data_ptr(), nsv, wsb.data_ptr(), nb, st)
    torch.cuda.synchronize()
    return outs + [dx]


def test_backward_ignores_unwritten_slot_contents():
    """Slots filled with NaN past the S written positions (S 200 in 512-position slots):
    the training forward and backward give the zero-filled results bit for bit."""
    w = small_workload("bwd-garbage", 3, 512, 4, 2, [0, 0, 2], seed=24)
    say("[backward garbage] S=200 cap=512")
    a = _train_outputs(w, 2, 200, 512, 0.0)
    b = _train_outputs(w, 2, 200, 512, float("nan"))
    for i, (u, v) in enumerate(zip(a, b)):
        assert bool(torch.isfinite(v.float()).all().item()), i
        assert torch.equal(u, v), i
    say("  bit-identical")
