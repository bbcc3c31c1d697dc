"""GPU parity through the C ABI against the fp64 oracle, at sizes the oracle
finishes in seconds: several tiles plus ragged tails, GQA ratios 1/2/4/8,
producer and consumer layers, prefill and decode, bf16 and fp32."""
import numpy as np
import pytest
import torch

import kvp_inputs as ki
from kvp_inputs import device as kd
from oracle import attention as oat
from paper_2608_15943_amd import binding as kb

from gpu_util import (DEV, build_device_model, oracle_weights, rel_err, run_prefill, say,
                      small_workload, tdtype, to_np, tol, workspace)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    kb.lib()


def test_device_generator_matches_host():
    w = ki.stage_share_prefill()
    t = torch.empty((w.a * w.d_h, w.h), dtype=torch.bfloat16, device=DEV)
    kd.fill_weight(w, ki.KIND_WQ, 3, t.data_ptr())
    host = ki.weight(w, ki.KIND_WQ, 3)
    assert np.array_equal(t.float().cpu().numpy(), host)
    x = torch.empty((2, 100, w.h), dtype=torch.bfloat16, device=DEV)
    kd.fill_prefill_x(w, x.data_ptr(), 2, 100)
    assert np.array_equal(x[1].float().cpu().numpy(), ki.prefill_x(w, [1], np.arange(100))[0])
    K = torch.empty((2, w.g, 192, w.d_h), dtype=torch.bfloat16, device=DEV)
    V = torch.empty((2, w.g, w.d_h, 192), dtype=torch.bfloat16, device=DEV)
    kd.fill_cache(w, 2, K.data_ptr(), V.data_ptr(), 2, 192, 150)
    hk = ki.cache_contents(w, ki.KIND_KCACHE, 2, 1, 150)
    hv = ki.cache_contents(w, ki.KIND_VCACHE, 2, 1, 150)
    assert np.array_equal(K[1, :, :150].float().cpu().numpy(), hk)
    assert np.array_equal(V[1, :, :, :150].float().cpu().numpy().transpose(0, 2, 1), hv)


def _prefill_case(w, B, S, cap):
    say(f"[prefill] {w.name} B={B} S={S} tau={w.tau}")
    dm = build_device_model(w, B, S, cap)
    x, y = run_prefill(dm, B, S)
    ws = oracle_weights(w)
    worst = 0.0
    for b in range(B):
        xb = ki.prefill_x(w, [b], np.arange(S))[0]
        ref, _, _, caches = oat.stack_prefill(xb, ws, w.tau, w.a, w.g, w.d_h, w.rope_base)
        e = rel_err(to_np(y[b]), ref)
        worst = max(worst, e)
        assert e <= tol(w), (b, e)
        for p, (K, V) in dm.slots.items():
            ek = rel_err(to_np(K[b, :, :S]), caches[p][0])
            ev = rel_err(to_np(V[b, :, :, :S]).transpose(0, 2, 1), caches[p][1])
            assert ek <= tol(w) and ev <= tol(w), (p, ek, ev)
    say(f"  max rel err {worst:.3e}")


def test_tiny_fp32_stack():
    w = ki.tiny_fp32()
    _prefill_case(w, 1, 128, 128)


def test_fp32_ragged_two_sequences():
    w = small_workload("fp32-gqa", 3, 256, 4, 2, [0, 0, 2], dtype="fp32", d_h=64)
    _prefill_case(w, 2, 77, 96)


@pytest.mark.parametrize("h,a,g,tau,B,S", [
    (256, 2, 2, [0, 0], 1, 64),              # MHA, one tile
    (512, 4, 2, [0, 1, 1, 3], 2, 200),       # GQA r=2, ragged S, chain map
    (512, 4, 1, [0, 0, 0], 1, 333),          # r=4, consumers only after layer 0
    (1024, 8, 1, [0, 0], 1, 130),            # r=8, S just past a query tile
    (256, 2, 1, [0, 1], 3, 1),               # S = 1
    (256, 2, 1, [0, 1], 5, 3),               # S < 4: one 4-row group spans sequences
    (512, 4, 2, [0, 0, 2], 4, 300),          # B*g = 8: whole KV-head groups per XCD
    (512, 4, 4, [0, 1], 4, 520),             # B*g = 16, r=1, three query tiles
])
def test_bf16_stack(h, a, g, tau, B, S):
    w = small_workload(f"bf16-h{h}-a{a}-g{g}", len(tau), h, a, g, tau)
    cap = ((S + 63) // 64) * 64 + 64
    _prefill_case(w, B, S, cap)


def test_bf16_stack_capacity_equals_length():
    """kv_capacity == S with S % 128 == 64: the last 128-position key tile of the
    prefill attention runs past the slot and must not read or use anything there."""
    w = small_workload("bf16-h512-a4-g2-capS", 3, 512, 4, 2, [0, 0, 2])
    _prefill_case(w, 2, 320, 320)


def test_bf16_layer_forward_producer_then_consumer():
    """kvp_layer_forward on seeded inputs: attention output and residual per layer."""
    w = small_workload("bf16-layers", 2, 512, 4, 2, [0, 0])
    B, S, cap = 2, 150, 192
    dm = build_device_model(w, B, S, cap)
    ws_t, n = workspace(dm, kb.KVP_PHASE_PREFILL, B, S)
    st = torch.cuda.current_stream().cuda_stream
    oracle_w = oracle_weights(w)
    kv = {}
    for l in range(2):
        x = torch.empty((B, S, w.h), dtype=torch.bfloat16, device=DEV)
        wl = ki.Workload(**{**w.__dict__, "seed": 100 + l})   # a fresh seeded input per layer
        kd.fill_prefill_x(wl, x.data_ptr(), B, S)
        o = torch.empty((B, S, w.a * w.d_h), dtype=torch.bfloat16, device=DEV)
        y = torch.empty_like(x)
        dm.model.kvp_layer_forward(l, x.data_ptr(), o.data_ptr(), y.data_ptr(), B, S,
                                   ws_t.data_ptr(), n, st)
        torch.cuda.synchronize()
        for b in range(B):
            xb = ki.prefill_x(wl, [b], np.arange(S))[0]
            shared = kv.get(b) if l == 1 else None
            yr, orf, kvb = oat.layer_prefill(xb, oracle_w[l], w.a, w.g, w.d_h, w.rope_base,
                                            shared_kv=shared)
            if l == 0:
                kv[b] = kvb
            assert rel_err(to_np(o[b]), orf) <= 2e-2
            assert rel_err(to_np(y[b]), yr) <= 2e-2


def _decode_case(w, B, lens, cap):
    say(f"[decode] {w.name} B={B} lens={list(lens)} tau={w.tau}")
    npos = int(max(lens))
    dm = build_device_model(w, B, 1, cap, fill_cache_npos=max(npos, 1))
    x = torch.empty((B, w.h), dtype=tdtype(w), device=DEV)
    kd.fill_decode_x(w, x.data_ptr(), B)
    y = torch.empty_like(x)
    lens_t = torch.tensor(lens, dtype=torch.int32, device=DEV)
    ws_t, n = workspace(dm, kb.KVP_PHASE_DECODE, B)
    dm.model.kvp_decode_step(x.data_ptr(), lens_t.data_ptr(), npos, y.data_ptr(), B,
                             ws_t.data_ptr(), n, torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    ows = oracle_weights(w)
    xs = ki.decode_x(w, list(range(B)))
    worst = 0.0
    for b in range(B):
        L = int(lens[b])
        caches = {p: (ki.cache_contents(w, ki.KIND_KCACHE, p, b, L),
                      ki.cache_contents(w, ki.KIND_VCACHE, p, b, L)) for p in dm.slots}
        yr, _, new_kv = oat.decode_step(xs[b], L, ows, w.tau, caches, w.a, w.g, w.d_h, w.rope_base)
        e = rel_err(to_np(y[b]), yr)
        worst = max(worst, e)
        assert e <= tol(w), (b, e)
        for p, (K, V) in dm.slots.items():
            assert rel_err(to_np(K[b, :, L]), new_kv[p][0]) <= tol(w)
            assert rel_err(to_np(V[b, :, :, L]), new_kv[p][1]) <= tol(w)
    say(f"  max rel err {worst:.3e}")


def test_decode_fp32_tiny():
    w = ki.tiny_fp32()
    _decode_case(w, 2, [0, 100], 128)


@pytest.mark.parametrize("h,a,g,tau,lens,cap", [
    (512, 4, 1, [0, 0, 2, 2], [0, 1, 63, 64], 128),          # r=4, tile edges
    (512, 4, 2, [0, 0, 0], [300, 1000, 257], 1024),           # r=2, several splits
    (1024, 8, 8, [0, 1], [2000], 2048),                       # MHA
    (512, 4, 1, [0, 0], [5000, 3, 4095], 5120),                # ragged, > 1 split
    (512, 4, 2, [0, 0, 2], [127, 0, 64, 1], 128),             # new token in the slot's last position
    # 37 sequences: above the fused small-batch projections, so the split-K projection kernels
    # run with a partial 16-row block (rows 32-36 of 48)
    (512, 4, 2, [0, 0, 2], [(37 * i) % 301 for i in range(37)], 384),
    # d_model 8192 (K = 8192): fused projections with 16 waves per workgroup, and split-K
    (8192, 64, 8, [0, 0], [5, 70, 130], 192),
    (8192, 64, 8, [0, 0], [(41 * i + 3) % 180 for i in range(20)], 192),
])
def test_decode_bf16(h, a, g, tau, lens, cap):
    w = small_workload(f"dec-h{h}-a{a}-g{g}", len(tau), h, a, g, tau)
    _decode_case(w, len(lens), lens, cap)


def test_decode_fused_projections_equal_split_k():
    """Batches of up to 16 sequences run each projection as one fused kernel, larger ones as
    split-K partial sums plus epilogue kernels; both add the K slices in the same order, so a
    sequence's outputs and appended K/V are the same bits whichever path its batch takes.
    Sequence b's input and caches do not depend on the batch size: the first 16 sequences of
    a 17-sequence call (split-K) must equal a 16-sequence call (fused) bit for bit."""
    w = small_workload("dec-fused-vs-split", 3, 512, 4, 2, [0, 0, 2])
    cap = 384
    lens17 = [(53 * i + 11) % 300 for i in range(17)]
    out = {}
    for B in (16, 17):
        lens = lens17[:B]
        dm = build_device_model(w, B, 1, cap, fill_cache_npos=max(lens))
        x = torch.empty((B, w.h), dtype=tdtype(w), device=DEV)
        kd.fill_decode_x(w, x.data_ptr(), B)
        y = torch.empty_like(x)
        lens_t = torch.tensor(lens, dtype=torch.int32, device=DEV)
        ws_t, n = workspace(dm, kb.KVP_PHASE_DECODE, B)
        dm.model.kvp_decode_step(x.data_ptr(), lens_t.data_ptr(), max(lens), y.data_ptr(), B,
                                 ws_t.data_ptr(), n, torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
        kv = {p: (torch.stack([K[b, :, lens[b]] for b in range(16)]),
                  torch.stack([V[b, :, :, lens[b]] for b in range(16)])) for p, (K, V) in dm.slots.items()}
        out[B] = (y[:16].clone(), kv)
        del dm, x, y, ws_t
    assert torch.equal(out[16][0], out[17][0])
    for p in out[16][1]:
        assert torch.equal(out[16][1][p][0], out[17][1][p][0])
        assert torch.equal(out[16][1][p][1], out[17][1][p][1])


def test_identity_map_equals_unshared_run_of_same_weights():
    """A shared map and the identity map differ only in which K/V a layer reads."""
    w = small_workload("map-vs-identity", 2, 512, 4, 2, [0, 0])
    wi = w.with_map([0, 1])
    B, S = 1, 96
    y_shared = run_prefill(build_device_model(w, B, S, 128), B, S)[1]
    y_ident = run_prefill(build_device_model(wi, B, S, 128), B, S)[1]
    ws = oracle_weights(wi)
    xb = ki.prefill_x(w, [0], np.arange(S))[0]
    ref_i = oat.stack_prefill(xb, ws, [0, 1], w.a, w.g, w.d_h, w.rope_base)[0]
    ref_s = oat.stack_prefill(xb, oracle_weights(w), [0, 0], w.a, w.g, w.d_h, w.rope_base)[0]
    assert rel_err(to_np(y_ident[0]), ref_i) <= 2e-2
    assert rel_err(to_np(y_shared[0]), ref_s) <= 2e-2
    assert rel_err(to_np(y_shared[0]), to_np(y_ident[0])) > 1e-2


def test_debug_sync_mode_gives_the_same_results():
    """A context created with KVP_DEBUG_SYNC set waits for and checks every launch; prefill
    and decode results are bit-identical to a normal context's."""
    import os
    w = small_workload("debug-sync", 3, 512, 4, 2, [0, 0, 2], seed=41)
    B, S, cap = 2, 150, 256
    outs = []
    for flag in ("0", "1"):
        os.environ["KVP_DEBUG_SYNC"] = flag
        try:
            dm = build_device_model(w, B, S, cap)
        finally:
            os.environ.pop("KVP_DEBUG_SYNC", None)
        _, y = run_prefill(dm, B, S)
        x = torch.empty((B, w.h), dtype=torch.bfloat16, device=DEV)
        kd.fill_decode_x(w, x.data_ptr(), B)
        yd = torch.empty_like(x)
        lens = torch.tensor([S, S - 7], dtype=torch.int32, device=DEV)
        ws_t, n = workspace(dm, kb.KVP_PHASE_DECODE, B)
        dm.model.kvp_decode_step(x.data_ptr(), lens.data_ptr(), S, yd.data_ptr(), B, ws_t.data_ptr(), n,
                                 torch.cuda.current_stream().cuda_stream)
        torch.cuda.synchronize()
        outs.append((y, yd, [t.clone() for kv in dm.slots.values() for t in kv]))
    assert torch.equal(outs[0][0], outs[1][0]) and torch.equal(outs[0][1], outs[1][1])
    for a_, b_ in zip(outs[0][2], outs[1][2]):
        assert torch.equal(a_, b_)
    say("  debug-sync results bit-identical")
