"""kvp_decode_step_noalloc (workspace in the library's static device array) against
kvp_decode_step (caller workspace) through the C ABI: two calls in a row, the second with a
smaller batch and other lengths, on two device models built from the same seeded inputs;
the outputs and every producer's cache must be bit-identical after each call (same kernels,
same arithmetic; the second call also shows that nothing left in the array by the first
leaks into the result)."""
import numpy as np
import pytest
import torch

import kvp_inputs as ki
from kvp_inputs import device as kd
from oracle import attention as oat
from paper_2608_15943_amd import binding as kb

from gpu_util import DEV, build_device_model, oracle_weights, rel_err, say, small_workload, tdtype, to_np, \
    workspace
from gpu_util import tol as tol_for

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    kb.lib()


def _lens(seed, B, hi):
    return [int(v) for v in np.random.default_rng(seed).integers(0, hi, size=B)]


CASES = [
    # name, L, h, a, g, tau, dtype, d_h, cap, first lens, second lens
    ("bf16-r2", 3, 512, 4, 2, [0, 0, 2], "bf16", 128, 1024,
     [300, 0, 1000, 64, 5, 777], [10, 1022, 128]),
    ("bf16-d4096-b64", 2, 4096, 32, 8, [0, 0], "bf16", 128, 2048,
     _lens(1, 64, 2047), _lens(2, 8, 2047)),
    ("fp32-tiny", 4, 256, 4, 4, [0, 0, 2, 2], "fp32", 64, 128, [100, 3, 0], [127]),
]


@pytest.mark.parametrize("name,L,h,a,g,tau,dtype,d_h,cap,lens1,lens2", CASES)
def test_noalloc_decode_equals_decode_step(name, L, h, a, g, tau, dtype, d_h, cap, lens1, lens2):
    w = small_workload(f"noalloc-{name}", L, h, a, g, tau, dtype=dtype, d_h=d_h, seed=31)
    Bmax = max(len(lens1), len(lens2))
    say(f"[noalloc] {w.name} B={len(lens1)} then {len(lens2)} cap={cap}")
    npos = cap - 1
    dm_ref = build_device_model(w, Bmax, 1, cap, fill_cache_npos=npos)
    dm_new = build_device_model(w, Bmax, 1, cap, fill_cache_npos=npos)
    st = torch.cuda.current_stream().cuda_stream
    for call, lens in enumerate((lens1, lens2)):
        B = len(lens)
        x = torch.empty((B, w.h), dtype=tdtype(w), device=DEV)
        kd.fill_decode_x(w, x.data_ptr(), B)
        lens_t = torch.tensor(lens, dtype=torch.int32, device=DEV)
        y_ref = torch.empty_like(x)
        y_new = torch.full_like(x, float("nan"))
        ws_t, n = workspace(dm_ref, kb.KVP_PHASE_DECODE, B)
        dm_ref.model.kvp_decode_step(x.data_ptr(), lens_t.data_ptr(), max(lens), y_ref.data_ptr(), B,
                                     ws_t.data_ptr(), n, st)
        dm_new.model.kvp_decode_step_noalloc(x.data_ptr(), lens_t.data_ptr(), max(lens), y_new.data_ptr(), B, st)
        torch.cuda.synchronize()
        assert torch.equal(y_ref, y_new), f"call {call}: outputs differ"
        for p in dm_ref.slots:
            assert torch.equal(dm_ref.slots[p][0], dm_new.slots[p][0]), f"call {call}: K slot {p}"
            assert torch.equal(dm_ref.slots[p][1], dm_new.slots[p][1]), f"call {call}: V slot {p}"
        say(f"  call {call} (B={B}): bit-identical outputs and caches")
    # The second call's last sequence against the oracle, which replays both calls for it
    # (the first call appended K/V at lens1[b], which the second may read).
    b = len(lens2) - 1
    ows = oracle_weights(w)
    hi = max(lens2[b], lens1[b] if b < len(lens1) else 0)
    caches = {p: (ki.cache_contents(w, ki.KIND_KCACHE, p, b, hi + 1), ki.cache_contents(w, ki.KIND_VCACHE, p, b, hi + 1))
              for p in dm_new.slots}
    caches = {p: (np.array(k, dtype=np.float64), np.array(v, dtype=np.float64)) for p, (k, v) in caches.items()}
    xb = ki.decode_x(w, [b])[0]
    if b < len(lens1):
        _, _, new_kv = oat.decode_step(xb, lens1[b], ows, w.tau, caches, w.a, w.g, w.d_h, w.rope_base)
        for p, (kn, vn) in new_kv.items():
            caches[p][0][:, lens1[b]] = kn
            caches[p][1][:, lens1[b]] = vn
    yr, _, _ = oat.decode_step(xb, lens2[b], ows, w.tau, caches, w.a, w.g, w.d_h, w.rope_base)
    e = rel_err(to_np(y_new[b]), yr)
    say(f"  sequence {b} of the second call against the oracle: {e:.3e}")
    assert e <= tol_for(w)
