"""GPU tests of paged KV storage (kvp_set_kv_pool, kvp_prefill_paged, kvp_decode_step_paged).

The paged calls run the same kernels and arithmetic as the contiguous slots, only the
addresses of K and V differ, so the outputs are compared bit for bit with the slot path
(which the parity tests compare with the oracle), the pages' contents with the slots', and
the small cases directly with the oracle as well.  Page tables are scattered (a seeded
permutation of the pool), so every 64-position tile comes from an unrelated page."""
import numpy as np
import pytest
import torch

import kvp_inputs as ki
from kvp_inputs import device as kd
from oracle import attention as oat
from paper_2608_15943_amd import binding as kb

from gpu_util import (DEV, build_device_model, oracle_weights, rel_err, say, small_workload, to_np,
                      workspace)

pytestmark = pytest.mark.gpu
PAGE = 64


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    kb.lib()


def scattered_table(npos, stride, spare, seed):
    """Table [B][stride] mapping ceil(npos_b / 64) pages per sequence to a seeded random
    choice of distinct pages of a pool with `spare` extra pages; -1 elsewhere."""
    need = [(int(n) + PAGE - 1) // PAGE for n in npos]
    n_pages = sum(need) + spare
    perm = np.random.RandomState(seed).permutation(n_pages).astype(np.int32)
    tab = np.full((len(npos), stride), -1, dtype=np.int32)
    k = 0
    for b, n in enumerate(need):
        assert n <= stride
        tab[b, :n] = perm[k:k + n]
        k += n
    return tab, n_pages


def make_pools(dm, n_pages):
    w = dm.w
    pools = {}
    for l in range(w.L):
        if w.tau[l] == l:
            K = torch.zeros((w.g, n_pages, PAGE, w.d_h), dtype=torch.bfloat16, device=DEV)
            V = torch.zeros((w.g, n_pages, w.d_h, PAGE), dtype=torch.bfloat16, device=DEV)
            dm.model.kvp_set_kv_pool(l, K.data_ptr(), V.data_ptr(), n_pages)
            pools[l] = (K, V)
    return pools


def gather(pools, tab_t, b, npos):
    """Logical K [g][npos][d] and V^T [g][d][npos] of sequence b, read back from the pages."""
    out = {}
    idx = torch.arange(npos, device=DEV)
    pg = tab_t[b].long()[idx // PAGE]
    row = idx % PAGE
    for l, (K, V) in pools.items():
        out[l] = (K[:, pg, row, :], V[:, pg, :, row].permute(1, 2, 0))
    return out


@pytest.mark.parametrize("h,a,g,tau,lens,stride", [
    (512, 4, 1, [0, 0, 2], [0, 1, 63, 64, 200, 130], 4),     # r = 4, tile and page edges
    (512, 4, 2, [0, 0, 0], [300, 1000, 257], 17),            # r = 2, several splits, spare row
    (512, 4, 2, [0, 0, 2], [127, 0, 255], 4),                # new token in the row's last page
    # 37 sequences: the split-K projections with their epilogue appending through the table
    (512, 4, 2, [0, 0, 2], [(29 * i + 5) % 260 for i in range(37)], 5),
])
def test_decode_paged_equals_slots(h, a, g, tau, lens, stride):
    w = small_workload(f"paged-dec-h{h}-a{a}-g{g}", len(tau), h, a, g, tau, seed=31)
    B = len(lens)
    say(f"[paged decode] {w.name} lens={lens} stride={stride}")
    npos = int(max(lens))
    cap = PAGE * stride
    dm = build_device_model(w, B, 1, cap, fill_cache_npos=max(npos, 1))
    tab, n_pages = scattered_table([n + 1 for n in lens], stride, 5, seed=7)
    pools = make_pools(dm, n_pages)
    tab_t = torch.from_numpy(tab).to(DEV)
    lens_t = torch.tensor(lens, dtype=torch.int32, device=DEV)
    for l in pools:
        kd.fill_cache_pages(w, l, pools[l][0].data_ptr(), pools[l][1].data_ptr(), tab_t.data_ptr(), stride,
                            n_pages, lens_t.data_ptr(), B)
    x = torch.empty((B, w.h), dtype=torch.bfloat16, device=DEV)
    kd.fill_decode_x(w, x.data_ptr(), B)
    y_c = torch.empty_like(x)
    y_p = torch.full_like(x, float("nan"))
    ws, n = workspace(dm, kb.KVP_PHASE_DECODE, B)
    st = torch.cuda.current_stream().cuda_stream
    dm.model.kvp_decode_step(x.data_ptr(), lens_t.data_ptr(), npos, y_c.data_ptr(), B, ws.data_ptr(), n, st)
    dm.model.kvp_decode_step_paged(x.data_ptr(), lens_t.data_ptr(), npos, tab_t.data_ptr(), stride,
                                   y_p.data_ptr(), B, ws.data_ptr(), n, st)
    torch.cuda.synchronize()
    assert torch.equal(y_c, y_p), "paged decode differs from the slot path"
    ows = oracle_weights(w)
    xs = ki.decode_x(w, list(range(B)))
    for b in range(B):
        L = lens[b]
        got = gather(pools, tab_t, b, L + 1)
        for l, (K, V) in dm.slots.items():
            # Pages hold the filled positions and the appended one exactly as the slot does.
            assert torch.equal(got[l][0], K[b, :, :L + 1]), (b, l, "K")
            assert torch.equal(got[l][1], V[b, :, :, :L + 1]), (b, l, "V")
        caches = {p: (ki.cache_contents(w, ki.KIND_KCACHE, p, b, L),
                      ki.cache_contents(w, ki.KIND_VCACHE, p, b, L)) for p in dm.slots}
        yr = oat.decode_step(xs[b], L, ows, w.tau, caches, w.a, w.g, w.d_h, w.rope_base)[0]
        assert rel_err(to_np(y_p[b]), yr) <= 2e-2, b
    say("  bit-identical to the slots; oracle ok")


@pytest.mark.parametrize("B,S,stride", [(2, 200, 4), (1, 128, 2), (3, 1, 1), (1, 333, 9)])
def test_prefill_paged_equals_slots(B, S, stride):
    w = small_workload("paged-pre", 3, 512, 4, 2, [0, 0, 2], seed=32)
    say(f"[paged prefill] B={B} S={S} stride={stride}")
    cap = (S + 63) // 64 * 64
    dm = build_device_model(w, B, S, cap)
    tab, n_pages = scattered_table([S] * B, stride, 3, seed=8)
    pools = make_pools(dm, n_pages)
    tab_t = torch.from_numpy(tab).to(DEV)
    x = torch.empty((B, S, w.h), dtype=torch.bfloat16, device=DEV)
    kd.fill_prefill_x(w, x.data_ptr(), B, S)
    y_c = torch.empty_like(x)
    y_p = torch.full_like(x, float("nan"))
    ws, n = workspace(dm, kb.KVP_PHASE_PREFILL, B, S)
    st = torch.cuda.current_stream().cuda_stream
    dm.model.kvp_prefill(x.data_ptr(), y_c.data_ptr(), B, S, ws.data_ptr(), n, st)
    dm.model.kvp_prefill_paged(x.data_ptr(), y_p.data_ptr(), B, S, tab_t.data_ptr(), stride, ws.data_ptr(), n, st)
    torch.cuda.synchronize()
    assert torch.equal(y_c, y_p), "paged prefill differs from the slot path"
    ows = oracle_weights(w)
    for b in range(B):
        got = gather(pools, tab_t, b, S)
        for l, (K, V) in dm.slots.items():
            assert torch.equal(got[l][0], K[b, :, :S]), (b, l, "K")
            assert torch.equal(got[l][1], V[b, :, :, :S]), (b, l, "V")
        xb = ki.prefill_x(w, [b], np.arange(S))[0]
        ref = oat.stack_prefill(xb, ows, w.tau, w.a, w.g, w.d_h, w.rope_base)[0]
        assert rel_err(to_np(y_p[b]), ref) <= 2e-2, b
    say("  bit-identical to the slots; oracle ok")


def test_decode_128k_ragged_paged_full_size():
    """The ragged decode configuration (32 layers, d_model 4096, 32 / 8 heads, B 8, contexts
    64K-128K, groups of 4 layers share) on scattered pages: bit-identical to the slots."""
    w = ki.decode_128k_ragged()
    lens = w.lengths()
    B = w.batch
    stride = w.kv_capacity // PAGE
    say(f"[paged decode full] {w.name} lens {lens.min()}..{lens.max()}")
    npos = int(lens.max())
    dm = build_device_model(w, B, 1, w.kv_capacity, fill_cache_npos=npos)
    tab, n_pages = scattered_table([int(n) + 1 for n in lens], stride, 0, seed=9)
    pools = make_pools(dm, n_pages)
    tab_t = torch.from_numpy(tab).to(DEV)
    lens_t = torch.tensor(lens, dtype=torch.int32, device=DEV)
    for l in pools:
        kd.fill_cache_pages(w, l, pools[l][0].data_ptr(), pools[l][1].data_ptr(), tab_t.data_ptr(), stride,
                            n_pages, lens_t.data_ptr(), B)
    x = torch.empty((B, w.h), dtype=torch.bfloat16, device=DEV)
    kd.fill_decode_x(w, x.data_ptr(), B)
    y_c = torch.empty_like(x)
    y_p = torch.full_like(x, float("nan"))
    ws, n = workspace(dm, kb.KVP_PHASE_DECODE, B)
    st = torch.cuda.current_stream().cuda_stream
    dm.model.kvp_decode_step(x.data_ptr(), lens_t.data_ptr(), npos, y_c.data_ptr(), B, ws.data_ptr(), n, st)
    dm.model.kvp_decode_step_paged(x.data_ptr(), lens_t.data_ptr(), npos, tab_t.data_ptr(), stride,
                                   y_p.data_ptr(), B, ws.data_ptr(), n, st)
    torch.cuda.synchronize()
    assert torch.equal(y_c, y_p), "paged decode differs from the slot path at full size"
    for b in range(B):
        L = int(lens[b])
        idx = torch.tensor([L], device=DEV)
        pg = tab_t[b].long()[idx // PAGE]
        for l, (K, V) in dm.slots.items():
            Kp, Vp = pools[l]
            assert torch.equal(Kp[:, pg, idx % PAGE, :][:, 0], K[b, :, L]), (b, l)
            assert torch.equal(Vp[:, pg, :, idx % PAGE][0], V[b, :, :, L]), (b, l)
    say("  bit-identical to the slots, appended rows included")
    del dm, pools, x, y_c, y_p, ws
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def test_decode_batches_above_64_run_in_chunks():
    """B = 130 sequences (bf16 kernels take 64 per launch): one call on slots and one on
    scattered pages equal calls of at most 64 sequences bit for bit; sampled sequences
    match the oracle."""
    w = small_workload("dec-b130", 3, 512, 4, 2, [0, 0, 2], seed=33)
    B, stride = 130, 2
    lens = [(37 * b) % 120 for b in range(B)]
    say(f"[decode B={B}] lens {min(lens)}..{max(lens)}")
    npos = int(max(lens))
    dm = build_device_model(w, B, 1, PAGE * stride, fill_cache_npos=max(npos, 1))
    tab, n_pages = scattered_table([n + 1 for n in lens], stride, 0, seed=10)
    pools = make_pools(dm, n_pages)
    tab_t = torch.from_numpy(tab).to(DEV)
    lens_t = torch.tensor(lens, dtype=torch.int32, device=DEV)
    for l in pools:
        kd.fill_cache_pages(w, l, pools[l][0].data_ptr(), pools[l][1].data_ptr(), tab_t.data_ptr(), stride,
                            n_pages, lens_t.data_ptr(), B)
    x = torch.empty((B, w.h), dtype=torch.bfloat16, device=DEV)
    kd.fill_decode_x(w, x.data_ptr(), B)
    ws, n = workspace(dm, kb.KVP_PHASE_DECODE, B)
    st = torch.cuda.current_stream().cuda_stream
    slots0 = {l: (K.clone(), V.clone()) for l, (K, V) in dm.slots.items()}
    y_all = torch.full_like(x, float("nan"))
    dm.model.kvp_decode_step(x.data_ptr(), lens_t.data_ptr(), npos, y_all.data_ptr(), B, ws.data_ptr(), n, st)
    yp_all = torch.full_like(x, float("nan"))
    dm.model.kvp_decode_step_paged(x.data_ptr(), lens_t.data_ptr(), npos, tab_t.data_ptr(), stride,
                                   yp_all.data_ptr(), B, ws.data_ptr(), n, st)
    torch.cuda.synchronize()
    # Restore the slots (the call appended at len_b) and run the chunks one call each, on
    # a model whose slots start at the chunk's first sequence.
    y_parts = torch.full_like(x, float("nan"))
    row = w.g * PAGE * stride * w.d_h * 2   # bytes of one sequence in a K (or V) slot, bf16
    for b0 in range(0, B, 64):
        Bc = min(64, B - b0)
        mc = kb.Model(w.L, w.h, w.a, w.g, w.d_h, kb.KVP_DTYPE_BF16, w.tau, max_batch=Bc, max_seq=1,
                      kv_capacity=PAGE * stride, rope_base=w.rope_base)
        for l in range(w.L):
            prod = w.tau[l] == l
            t = dm.tensors
            mc.kvp_set_layer(l, t[f"wq{l}"].data_ptr(), t[f"wk{l}"].data_ptr() if prod else 0,
                             t[f"wv{l}"].data_ptr() if prod else 0, t[f"wo{l}"].data_ptr())
            if prod:
                K, V = slots0[l]
                mc.kvp_set_kv_slot(l, K.data_ptr() + b0 * row, V.data_ptr() + b0 * row)
        nc = mc.kvp_workspace_size(kb.KVP_PHASE_DECODE, Bc)
        wsc = torch.empty(nc, dtype=torch.uint8, device=DEV)
        mc.kvp_decode_step(x[b0:].data_ptr(), lens_t[b0:].data_ptr(), npos, y_parts[b0:].data_ptr(), Bc,
                           wsc.data_ptr(), nc, st)
        torch.cuda.synchronize()
        mc.close()
    assert torch.equal(y_all, y_parts), "chunked decode differs from separate calls"
    assert torch.equal(y_all, yp_all), "paged chunked decode differs from the slots"
    ows = oracle_weights(w)
    for b in (0, 63, 64, 129):
        L = lens[b]
        caches = {p: (ki.cache_contents(w, ki.KIND_KCACHE, p, b, L),
                      ki.cache_contents(w, ki.KIND_VCACHE, p, b, L)) for p in dm.slots}
        yr = oat.decode_step(ki.decode_x(w, [b])[0], L, ows, w.tau, caches, w.a, w.g, w.d_h, w.rope_base)[0]
        assert rel_err(to_np(y_all[b]), yr) <= 2e-2, b
    say("  chunks bit-identical to separate calls and to pages; oracle ok")


def test_prefill_paged_full_size_stage():
    """The 8-layer stage share (d_model 2048, 16 / 8 heads, B 4, S 4096) on scattered pages:
    output and every producer's K/V bit-identical to the slot path."""
    w = ki.stage_share_prefill()
    B, S = w.batch, w.seq
    stride = S // PAGE
    say(f"[paged prefill full] {w.name}")
    dm = build_device_model(w, B, S, w.kv_capacity)
    tab, n_pages = scattered_table([S] * B, stride, 0, seed=11)
    pools = make_pools(dm, n_pages)
    tab_t = torch.from_numpy(tab).to(DEV)
    x = torch.empty((B, S, w.h), dtype=torch.bfloat16, device=DEV)
    kd.fill_prefill_x(w, x.data_ptr(), B, S)
    y_c = torch.empty_like(x)
    y_p = torch.full_like(x, float("nan"))
    ws, n = workspace(dm, kb.KVP_PHASE_PREFILL, B, S)
    st = torch.cuda.current_stream().cuda_stream
    dm.model.kvp_prefill(x.data_ptr(), y_c.data_ptr(), B, S, ws.data_ptr(), n, st)
    dm.model.kvp_prefill_paged(x.data_ptr(), y_p.data_ptr(), B, S, tab_t.data_ptr(), stride, ws.data_ptr(), n, st)
    torch.cuda.synchronize()
    assert torch.equal(y_c, y_p), "paged prefill differs from the slot path at full size"
    for b in range(B):
        got = gather(pools, tab_t, b, S)
        for l, (K, V) in dm.slots.items():
            assert torch.equal(got[l][0], K[b]), (b, l, "K")
            assert torch.equal(got[l][1], V[b]), (b, l, "V")
    say("  output and caches bit-identical to the slots")
    del dm, pools, x, y_c, y_p, ws
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def test_unwritten_cache_contents_are_never_used():
    """Cache memory past the written positions holds arbitrary bits in real use.  Slots and
    pools filled with NaN before a prefill (S 300 in 512-position slots / 5-page rows) and the
    decode step that follows give bit-identical results to zero-filled ones: positions >= S
    (or > len_b) only ever meet masks that select, never multiply."""
    w = small_workload("garbage-tail", 3, 512, 4, 2, [0, 0, 2], seed=34)
    B, S, cap, stride = 2, 300, 512, 8
    say(f"[garbage] B={B} S={S} cap={cap}")
    outs = {}
    for fill in (0.0, float("nan")):
        dm = build_device_model(w, B, S, cap)
        tab, n_pages = scattered_table([cap] * B, stride, 0, seed=12)
        pools = make_pools(dm, n_pages)
        for K, V in list(dm.slots.values()) + list(pools.values()):
            K.fill_(fill)
            V.fill_(fill)
        tab_t = torch.from_numpy(tab).to(DEV)
        x = torch.empty((B, S, w.h), dtype=torch.bfloat16, device=DEV)
        kd.fill_prefill_x(w, x.data_ptr(), B, S)
        y = torch.empty_like(x)
        yp = torch.empty_like(x)
        ws, n = workspace(dm, kb.KVP_PHASE_PREFILL, B, S)
        st = torch.cuda.current_stream().cuda_stream
        dm.model.kvp_prefill(x.data_ptr(), y.data_ptr(), B, S, ws.data_ptr(), n, st)
        dm.model.kvp_prefill_paged(x.data_ptr(), yp.data_ptr(), B, S, tab_t.data_ptr(), stride, ws.data_ptr(), n,
                                   st)
        xd = torch.empty((B, w.h), dtype=torch.bfloat16, device=DEV)
        kd.fill_decode_x(w, xd.data_ptr(), B)
        lens_t = torch.full((B,), S, dtype=torch.int32, device=DEV)
        yd = torch.empty_like(xd)
        ydp = torch.empty_like(xd)
        wsd, nd = workspace(dm, kb.KVP_PHASE_DECODE, B)
        dm.model.kvp_decode_step(xd.data_ptr(), lens_t.data_ptr(), S, yd.data_ptr(), B, wsd.data_ptr(), nd, st)
        dm.model.kvp_decode_step_paged(xd.data_ptr(), lens_t.data_ptr(), S, tab_t.data_ptr(), stride,
                                       ydp.data_ptr(), B, wsd.data_ptr(), nd, st)
        torch.cuda.synchronize()
        outs[fill == fill] = (y, yp, yd, ydp)
        assert all(bool(torch.isfinite(t.float()).all().item()) for t in (y, yp, yd, ydp)), fill
    for a, b in zip(outs[True], outs[False]):
        assert torch.equal(a, b)
    say("  NaN-filled caches give the zero-filled results bit for bit")
