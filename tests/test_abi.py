"""The C ABI library on the CPU: it loads, exports every symbol that
include/kvpipe.h declares, its planner reproduces the oracle bit for bit, and
its host-side argument checks return the documented status codes.  Nothing
here launches a GPU kernel."""
import os
import random
import re

import numpy as np
import pytest

from oracle import planner as opl
from paper_2608_15943_amd import binding as kb

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    names = []
    for fn in os.listdir(os.path.join(ROOT, "include")):
        if fn.endswith(".h"):
            src = open(os.path.join(ROOT, "include", fn)).read()
            src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
            names += re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(kvp_\w+)\s*\(", src, flags=re.M)
    return sorted(set(names))


def test_library_exports_every_declared_symbol():
    names = declared_functions()
    assert len(names) >= 16
    lib = kb.lib()
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(kb.EXPORTS) == names


def test_status_strings():
    assert kb.status_name(kb.KVP_E_BAD_MAP) == "KVP_E_BAD_MAP"
    assert kb.status_name(0) == "KVP_OK"


# ---------------------------------------------------------------------------
# Planner: C++ vs the oracle, same IEEE double operations in the same order.
# ---------------------------------------------------------------------------

def _compare_plans(stage, ff, fs, lm, eps, m=0, adm=None, alpha=-1.0):
    P = max(stage) + 1
    ref = opl.plan_fir(stage, P, ff, fs, lm, eps, m=m, admissible=adm, alpha=alpha)
    got = kb.kvp_plan_fir(stage, ff, fs, lm, eps, m=m, admissible=adm, alpha=alpha, P=P)
    assert got["z"] == ref.z
    assert got["stage_flops"] == ref.stage_flops          # exact, not approximate
    assert got["fir"] == ref.fir
    assert got["n_converted"] == ref.n_converted
    assert got["stop_reason"] == ref.stop_reason
    return got


def test_planner_llama2_pp8_matches_oracle_and_paper():
    f0, f1 = kb.kvp_layer_flops(1, 8192, 4096, 32, 32, ffn=11008, causal=True)
    assert (f0, f1) == tuple(float(v) for v in opl.layer_flops_prefill(1, 8192, 4096, 32, 32, ffn=11008))
    stage = [l // 4 for l in range(32)]
    lm = 2.0 * 8192 * 4096 * 32000
    got = _compare_plans(stage, [f0] * 32, [f1] * 32, lm, eps=0.02, m=4)
    assert [l + 1 for l in range(32) if got["z"][l]] == [29, 30, 31, 32]
    assert abs(got["fir"] - 1.00040391) < 2e-5


def test_planner_toys_and_guardrail():
    toy = [l // 3 for l in range(12)]
    _compare_plans(toy, [10] * 12, [7] * 12, 6, 0.01)
    _compare_plans(toy, [10] * 12, [7] * 12, 9, 0.01)
    got = _compare_plans(toy, [10] * 12, [4] * 12, 4, 0.01, m=3)
    assert [l for l in range(12) if got["z"][l]] == [5, 8, 11]
    _compare_plans(toy, [10] * 12, [9] * 12, 30, 0.01, adm=[False] * 11 + [True])
    _compare_plans([l // 4 for l in range(32)], [100.0] * 32, [90.0] * 32, 500.0, 0.001, alpha=0.5)


def test_planner_random_property():
    rng = random.Random(1234)
    for _ in range(300):
        L = rng.randint(1, 40)
        P = rng.randint(1, L)
        cuts = sorted(rng.sample(range(1, L), P - 1)) if P > 1 else []
        stage, s = [], 0
        for l in range(L):
            if s < len(cuts) and l >= cuts[s]:
                s += 1
            stage.append(s)
        ff = [rng.uniform(1e9, 1e12) for _ in range(L)]
        fs = [f * rng.uniform(0.5, 0.99) for f in ff]
        lm = rng.uniform(0, 5e12)
        eps = rng.choice([1e-6, 1e-3, 0.01, 0.05, 0.2])
        m = rng.randint(0, L)
        adm = [rng.random() < 0.8 for _ in range(L)] if rng.random() < 0.5 else None
        alpha = rng.choice([-1.0, 0.0, 0.25, 0.5, 0.9])
        _compare_plans(stage, ff, fs, lm, eps, m=m, adm=adm, alpha=alpha)


def test_fir_and_layer_flops_closed_forms():
    assert kb.kvp_fir([30, 30, 30, 36]) == 36 / 31.5
    f0, f1 = kb.kvp_layer_flops(64, 32768, 4096, 32, 8, phase=kb.KVP_PHASE_DECODE)
    assert (f0, f1) == tuple(float(v) for v in opl.layer_flops_decode(64, 32768, 4096, 32, 8))
    f0, f1 = kb.kvp_layer_flops(4, 4096, 2048, 16, 8, causal=False)
    assert f0 == 4 * 4 * 4096 * 2048 ** 2 + 4 * 4 * 4096 * 2048 ** 2 / 2 + 4 * 4 * 4096 ** 2 * 2048


def test_planner_rejections():
    with pytest.raises(kb.KvpError) as e:
        kb.kvp_plan_fir([0, 1, 1], [1, 1, 1], [0.5] * 3, 0, eps=0.0)
    assert e.value.code == kb.KVP_E_INVALID_ARG
    with pytest.raises(kb.KvpError):        # decreasing stage index
        kb.kvp_plan_fir([0, 1, 0], [1] * 3, [0.5] * 3, 0, eps=0.1, P=2)
    with pytest.raises(kb.KvpError):        # skipped stage
        kb.kvp_plan_fir([0, 2, 2], [1] * 3, [0.5] * 3, 0, eps=0.1, P=3)
    with pytest.raises(kb.KvpError):        # F(0) - F(1) <= 0 on an admissible layer
        kb.kvp_plan_fir([0, 1], [1, 1], [1, 1], 0, eps=0.1)
    with pytest.raises(kb.KvpError):        # P > L
        kb.kvp_plan_fir([0], [1], [0.5], 0, eps=0.1, P=2)


def _random_partition(rng, L, P):
    cuts = sorted(rng.sample(range(1, L), P - 1)) if P > 1 else []
    return [sum(1 for c in cuts if l >= c) for l in range(L)]


def test_placements_match_oracle():
    rng = random.Random(99)
    fns = {kb.KVP_PLACE_UNIFORM: opl.place_uniform,
           kb.KVP_PLACE_SYMMETRIC_BIPOLAR: opl.place_symmetric_bipolar}
    for _ in range(400):
        L = rng.randint(1, 48)
        P = rng.randint(1, min(L, 12))
        stage = _random_partition(rng, L, P) if rng.random() < 0.5 else [l * P // L for l in range(L)]
        k = rng.randint(0, L + 2)
        adm = [rng.random() < 0.75 for _ in range(L)] if rng.random() < 0.4 else None
        alpha = rng.choice([-1.0, 0.0, 0.3, 0.5, 0.95])
        for strat, fn in fns.items():
            ref = fn(stage, P, k, admissible=adm, alpha=alpha)
            got = kb.kvp_place(strat, stage, k, admissible=adm, alpha=alpha, P=P)
            assert got == (ref[0], ref[1], ref[2]), (strat, stage, k, adm, alpha)


def test_stage_flops_matches_oracle():
    rng = random.Random(7)
    for _ in range(100):
        L = rng.randint(1, 40)
        P = rng.randint(1, L)
        stage = _random_partition(rng, L, P)
        ff = [rng.uniform(1e9, 1e12) for _ in range(L)]
        fs = [f * rng.uniform(0.5, 0.99) for f in ff]
        z = [rng.randint(0, 1) for _ in range(L)]
        lm = rng.uniform(0, 5e12)
        assert kb.kvp_stage_flops(stage, ff, fs, z, lm, P=P) == opl.stage_flops(stage, P, ff, fs, z, lm)


def test_fir_table_reproducer_table2():
    """The FIR-table reproducer (C++ planner) against the oracle's strategy table and
    the FIRs Table 2 prints for LLaMA2-7B, PP = 8, S = 8K, 4 KV-sharing layers."""
    from paper_2608_15943_amd.fir_table import fir_table
    rows = {r["strategy"]: r for r in fir_table(eps=1e-4)}
    stage = [l // 4 for l in range(32)]
    f0, f1 = opl.layer_flops_prefill(1, 8192, 4096, 32, 32, ffn=11008)
    ref = opl.strategy_table(stage, 8, [f0] * 32, [f1] * 32, opl.mm_flops(8192, 4096, 32000), 4, 1e-4)
    for name, z, F, f in ref:
        assert rows[name]["layers"] == [l + 1 for l in range(32) if z[l]]
        assert rows[name]["stage_flops"] == F and rows[name]["fir"] == f
    printed = {"baseline": (1.119453925, 1e-9), "uniform": (1.103804831, 4e-5),
               "symmetric_bipolar": (1.068260764, 4e-5), "arch_balanced": (1.00040391, 2e-5)}
    for name, (v, tol) in printed.items():
        assert abs(rows[name]["fir"] - v) < tol, name
    assert rows["uniform"]["layers"] == [17, 22, 27, 32]


def test_placement_rejections():
    for args in ((7, [0, 1], 1), (kb.KVP_PLACE_UNIFORM, [0, 1], -1),
                 (kb.KVP_PLACE_UNIFORM, [0, 1, 0], 1), (kb.KVP_PLACE_SYMMETRIC_BIPOLAR, [0, 2, 2], 1)):
        with pytest.raises(kb.KvpError) as e:
            kb.kvp_place(*args)
        assert e.value.code == kb.KVP_E_INVALID_ARG
    with pytest.raises(kb.KvpError):        # P > L
        kb.kvp_place(kb.KVP_PLACE_UNIFORM, [0], 1, P=2)
    with pytest.raises(kb.KvpError):        # stage index out of range
        kb.kvp_stage_flops([0, 3], [1.0, 1.0], [0.5, 0.5], [0, 0], 0.0, P=2)


def test_maps():
    assert kb.kvp_map_from_mask([0, 0, 0, 0, 0, 1, 0, 1]) == [0, 1, 2, 3, 4, 4, 6, 6]
    assert kb.kvp_map_from_mask([0, 1, 1, 1]) == opl.map_from_mask([0, 1, 1, 1])
    with pytest.raises(kb.KvpError) as e:
        kb.kvp_map_from_mask([1, 0])
    assert e.value.code == kb.KVP_E_BAD_MAP
    assert kb.kvp_canonicalize_map([0, 0, 1, 2, 4]) == [0, 0, 0, 0, 4]
    for bad in ([1], [0, 2, 2], [0, -1]):
        with pytest.raises(kb.KvpError) as e:
            kb.kvp_canonicalize_map(bad)
        assert e.value.code == kb.KVP_E_BAD_MAP


# ---------------------------------------------------------------------------
# Context and host-side argument checks (no kernel launches).
# ---------------------------------------------------------------------------

def _model(**kw):
    args = dict(L=4, h=256, a=2, g=1, d_h=128, dtype=kb.KVP_DTYPE_BF16, tau=[0, 0, 2, 2],
                max_batch=2, max_seq=64, kv_capacity=128)
    args.update(kw)
    return kb.Model(**args)


def test_create_validates_shape_and_map():
    m = _model(tau=[0, 1, 1, 2])
    assert m.kvp_get_map() == [0, 1, 1, 1]          # chains resolved
    for kw, code in [(dict(tau=[1, 0, 2, 2]), kb.KVP_E_BAD_MAP),
                     (dict(tau=[0, 3, 2, 2]), kb.KVP_E_BAD_MAP),
                     (dict(d_h=64, a=4), kb.KVP_E_SHAPE),
                     (dict(kv_capacity=100), kb.KVP_E_SHAPE),
                     (dict(kv_capacity=1 << 23), kb.KVP_E_SHAPE),
                     (dict(g=3), kb.KVP_E_INVALID_ARG),
                     (dict(h=300), kb.KVP_E_INVALID_ARG),
                     (dict(max_seq=256), kb.KVP_E_INVALID_ARG),
                     (dict(dtype=7), kb.KVP_E_INVALID_ARG),
                     (dict(dtype=kb.KVP_DTYPE_FP32, d_h=48, a=4, h=192), kb.KVP_E_SHAPE)]:
        with pytest.raises(kb.KvpError) as e:
            _model(**kw)
        assert e.value.code == code, kw


def test_set_layer_and_slot_rules():
    m = _model()
    fake = 1 << 20                                    # never dereferenced on the host
    m.kvp_set_layer(0, fake, fake, fake, fake)
    with pytest.raises(kb.KvpError) as e:            # consumer with its own K/V weights
        m.kvp_set_layer(1, fake, fake, fake, fake)
    assert e.value.code == kb.KVP_E_INVALID_ARG
    with pytest.raises(kb.KvpError):                 # producer without Wk
        m.kvp_set_layer(2, fake, 0, fake, fake)
    with pytest.raises(kb.KvpError):                 # consumers own no slot
        m.kvp_set_kv_slot(1, fake, fake)
    with pytest.raises(kb.KvpError):                 # misaligned
        m.kvp_set_layer(1, fake + 2, 0, 0, fake)


def test_workspace_and_call_checks():
    m = _model()
    n = m.kvp_workspace_size(kb.KVP_PHASE_PREFILL, 2, 64)
    assert n > 2 * 64 * 256 * 2 * 3
    with pytest.raises(kb.KvpError) as e:
        m.kvp_workspace_size(kb.KVP_PHASE_PREFILL, 3, 64)
    assert e.value.code == kb.KVP_E_CAPACITY
    fake = 1 << 20
    with pytest.raises(kb.KvpError) as e:            # weights never set
        m.kvp_prefill(fake, fake * 2, 2, 64, fake * 4, n)
    assert e.value.code == kb.KVP_E_STATE
    with pytest.raises(kb.KvpError) as e:            # workspace too small
        m.kvp_prefill(fake, fake * 2, 2, 64, fake * 4, n - 1)
    assert e.value.code == kb.KVP_E_WORKSPACE
    with pytest.raises(kb.KvpError) as e:            # S > max_seq
        m.kvp_prefill(fake, fake * 2, 2, 65, fake * 4, n)
    assert e.value.code == kb.KVP_E_CAPACITY
    with pytest.raises(kb.KvpError) as e:            # aliasing x and y
        m.kvp_prefill(fake, fake, 2, 64, fake * 4, n)
    assert e.value.code == kb.KVP_E_INVALID_ARG
    nd = m.kvp_workspace_size(kb.KVP_PHASE_DECODE, 2)
    with pytest.raises(kb.KvpError) as e:            # position does not fit the slot
        m.kvp_decode_step(fake, fake * 8, 128, fake * 2, 2, fake * 4, nd)
    assert e.value.code == kb.KVP_E_CAPACITY
    with pytest.raises(kb.KvpError) as e:            # B > max_batch
        m.kvp_decode_step(fake, fake * 8, 10, fake * 2, 3, fake * 4, nd)
    assert e.value.code == kb.KVP_E_CAPACITY


def test_training_entry_points_host_checks():
    # bf16 model with one consumer; no device memory is touched by these checks.
    m = kb.Model(2, 256, 2, 1, 128, kb.KVP_DTYPE_BF16, [0, 0], max_batch=2, max_seq=200,
                 kv_capacity=256)
    n1 = m.kvp_train_saved_size(2, 200)
    # Per layer: Q, O, X [400][256] bf16 and the log-sum-exp [2][2][256] fp32.
    assert n1 == 2 * (3 * 400 * 256 * 2 + 2 * 2 * 256 * 4)
    assert m.kvp_workspace_size(kb.KVP_PHASE_BACKWARD, 2, 200) > 0
    with pytest.raises(kb.KvpError) as e:
        m.kvp_train_saved_size(3, 200)
    assert e.value.code == kb.KVP_E_CAPACITY
    with pytest.raises(kb.KvpError) as e:      # a consumer has no dW_K, dW_V
        m.kvp_set_layer_grads(1, 16, 32, 48, 64)
    assert e.value.code == kb.KVP_E_INVALID_ARG
    with pytest.raises(kb.KvpError):           # a producer needs them
        m.kvp_set_layer_grads(0, 16, 0, 0, 64)
    with pytest.raises(kb.KvpError) as e:      # gradient buffers never set
        m.kvp_backward(16, 32, 48, 2, 200, 64, n1, 80, 1 << 40)
    assert e.value.code == kb.KVP_E_STATE
    m.kvp_set_layer_grads(0, 16, 32, 48, 64)
    m.kvp_set_layer_grads(1, 16, 0, 0, 64)
    with pytest.raises(kb.KvpError) as e:      # dx aliases dy
        m.kvp_backward(16, 32, 32, 2, 200, 64, n1, 80, 1 << 40)
    assert e.value.code == kb.KVP_E_INVALID_ARG
    with pytest.raises(kb.KvpError) as e:      # short saved buffer
        m.kvp_backward(16, 32, 48, 2, 200, 64, n1 - 1, 80, 1 << 40)
    assert e.value.code == kb.KVP_E_WORKSPACE
    with pytest.raises(kb.KvpError) as e:      # short workspace
        m.kvp_backward(16, 32, 48, 2, 200, 64, n1, 80, 16)
    assert e.value.code == kb.KVP_E_WORKSPACE
    m.close()
    # fp32 models: Q, O, X [8][64] fp32 per layer, no saved log-sum-exp (it is recomputed).
    f = kb.Model(2, 64, 1, 1, 64, kb.KVP_DTYPE_FP32, [0, 0], max_batch=1, max_seq=8, kv_capacity=8)
    assert f.kvp_train_saved_size(1, 8) == 2 * 3 * 8 * 64 * 4
    # dO, dQKV (producer width), statistics, one dK/dV sum pair, RoPE table; each
    # piece rounded up to 256 bytes.
    assert f.kvp_workspace_size(kb.KVP_PHASE_BACKWARD, 1, 8) == (2048 + 6144 + 256 + 256 + 4096 + 2048)
    with pytest.raises(kb.KvpError) as e:
        f.kvp_train_saved_size(1, 9)
    assert e.value.code == kb.KVP_E_CAPACITY
    f.close()


def test_calibration_entry_points_reject_bad_arguments():
    """include/kvp_calib.h: argument checks happen on the host, before any launch."""
    L = kb.lib()
    import ctypes as C
    f = C.c_double()
    assert L.kvp_calib_mfma_bf16(0, C.c_void_p(16), C.byref(f), None) == kb.KVP_E_INVALID_ARG
    assert L.kvp_calib_mfma_bf16(3, C.c_void_p(16), C.byref(f), None) == kb.KVP_E_INVALID_ARG
    assert L.kvp_calib_mfma_bf16(2, None, C.byref(f), None) == kb.KVP_E_INVALID_ARG
    assert L.kvp_calib_stream_read(None, 65536, C.c_void_p(16), None) == kb.KVP_E_INVALID_ARG
    assert L.kvp_calib_stream_read(C.c_void_p(256), 1000, C.c_void_p(16), None) == kb.KVP_E_INVALID_ARG
    assert L.kvp_calib_stream_read(C.c_void_p(258), 65536, C.c_void_p(16), None) == kb.KVP_E_INVALID_ARG
    assert "kvp_calib_stream_read" in L.kvp_last_error().decode()


def test_pager_allocates_all_or_nothing_and_reuses_pages():
    """kvp_pager_*: lowest pages first from a fresh pager, all-or-nothing growth, release."""
    p = kb.Pager(10, 3, 4)
    assert p.free_pages() == 10
    p.reserve(0, 130)                       # 3 pages: 0, 1, 2
    assert p.rows([0]).tolist() == [[0, 1, 2, -1]]
    p.reserve(0, 128)                       # never shrinks
    assert p.rows([0]).tolist() == [[0, 1, 2, -1]]
    p.reserve(1, 64)                        # exactly one page
    assert p.rows([1])[0, 0] == 3
    assert not p.try_reserve(2, 5 * 64)     # beyond the row (4 pages): nothing reserved
    assert p.free_pages() == 6
    p.reserve(2, 4 * 64)
    assert p.free_pages() == 2
    assert not p.try_reserve(1, 4 * 64)     # 3 more pages needed, 2 free: nothing changes
    assert p.rows([1]).tolist() == [[3, -1, -1, -1]] and p.free_pages() == 2
    p.release(0)
    assert p.free_pages() == 5 and p.rows([0]).tolist() == [[-1] * 4]
    p.reserve(1, 4 * 64)                    # the released pages come back first, in order
    assert p.rows([1]).tolist() == [[3, 0, 1, 2]]
    with pytest.raises(kb.KvpError) as e:
        p.reserve(3, 1)
    assert e.value.code == kb.KVP_E_INVALID_ARG
    p.close()


def test_pager_random_operations_keep_pages_disjoint():
    rng = np.random.RandomState(3)
    n_pages, seqs, row = 200, 12, 40
    p = kb.Pager(n_pages, seqs, row)
    held = [0] * seqs
    for _ in range(2000):
        s = int(rng.randint(seqs))
        if rng.rand() < 0.2:
            p.release(s)
            held[s] = 0
            continue
        n = int(rng.randint(0, row * 64 + 200))
        need = (n + 63) // 64
        free_before = p.free_pages()
        okay = p.try_reserve(s, n)
        add = max(0, need - held[s])
        assert okay == (need <= row and add <= free_before)
        if okay:
            held[s] = max(held[s], need)
        tab = p.rows(list(range(seqs)))
        mapped = tab[tab >= 0]
        assert len(mapped) == sum(held) == n_pages - p.free_pages()
        assert len(np.unique(mapped)) == len(mapped)          # no page in two places
        assert mapped.max(initial=-1) < n_pages
        for t in range(seqs):                                   # rows are prefixes
            assert (tab[t, :held[t]] >= 0).all() and (tab[t, held[t]:] == -1).all()
    p.close()


def test_paged_entry_points_host_checks():
    m = kb.Model(2, 256, 2, 1, 128, kb.KVP_DTYPE_BF16, [0, 0], max_batch=2, max_seq=200,
                 kv_capacity=256)
    assert m.kvp_page_bytes() == 2 * 64 * 1 * 128 * 2
    fake = 1 << 20
    with pytest.raises(kb.KvpError) as e:            # consumer owns no pool
        m.kvp_set_kv_pool(1, fake, fake, 4)
    assert e.value.code == kb.KVP_E_INVALID_ARG
    with pytest.raises(kb.KvpError) as e:
        m.kvp_set_kv_pool(0, fake, fake, 0)
    assert e.value.code == kb.KVP_E_INVALID_ARG
    m.kvp_set_layer(0, fake, fake, fake, fake)
    m.kvp_set_layer(1, fake, 0, 0, fake)
    n = m.kvp_workspace_size(kb.KVP_PHASE_PREFILL, 2, 200)
    with pytest.raises(kb.KvpError) as e:            # pools never set
        m.kvp_prefill_paged(fake, fake * 2, 2, 200, fake * 3, 4, fake * 4, n)
    assert e.value.code == kb.KVP_E_STATE
    m.kvp_set_kv_pool(0, fake, fake, 8)
    with pytest.raises(kb.KvpError) as e:            # S beyond the table's reach
        m.kvp_prefill_paged(fake, fake * 2, 2, 200, fake * 3, 3, fake * 4, n)
    assert e.value.code == kb.KVP_E_CAPACITY
    with pytest.raises(kb.KvpError) as e:            # no table
        m.kvp_prefill_paged(fake, fake * 2, 2, 200, 0, 4, fake * 4, n)
    assert e.value.code == kb.KVP_E_INVALID_ARG
    nd = m.kvp_workspace_size(kb.KVP_PHASE_DECODE, 2)
    with pytest.raises(kb.KvpError) as e:            # position 256 beyond a 4-page row
        m.kvp_decode_step_paged(fake, fake * 8, 256, fake * 3, 4, fake * 2, 2, fake * 4, nd)
    assert e.value.code == kb.KVP_E_CAPACITY
    m.close()
    f = kb.Model(1, 64, 1, 1, 64, kb.KVP_DTYPE_FP32, [0], max_batch=1, max_seq=8, kv_capacity=8)
    with pytest.raises(kb.KvpError) as e:
        f.kvp_set_kv_pool(0, fake, fake, 4)
    assert e.value.code == kb.KVP_E_SHAPE
    f.close()


def test_noalloc_decode_rejects_workspace_beyond_the_static_array():
    """kvp_decode_step_noalloc checks, before touching the GPU, that the call's workspace fits
    the library's 64 MiB device array: a 70B-wide model (d_model 8192) fits at B = 64 and not
    at B = 100; a NULL context or B < 1 is rejected as an argument error."""
    m = kb.Model(1, 8192, 64, 8, 128, kb.KVP_DTYPE_BF16, [0], max_batch=128, max_seq=1, kv_capacity=128)
    assert m.kvp_workspace_size(kb.KVP_PHASE_DECODE, 64) <= 64 << 20
    assert m.kvp_workspace_size(kb.KVP_PHASE_DECODE, 100) > 64 << 20
    fake = 1 << 20
    with pytest.raises(kb.KvpError) as e:
        m.kvp_decode_step_noalloc(fake, fake * 2, 10, fake * 4, 100)
    assert e.value.code == kb.KVP_E_WORKSPACE
    assert "static array" in kb.lib().kvp_last_error().decode()
    with pytest.raises(kb.KvpError) as e:
        m.kvp_decode_step_noalloc(fake, fake * 2, 10, fake * 4, 0)
    assert e.value.code == kb.KVP_E_INVALID_ARG
    assert kb.lib().kvp_decode_step_noalloc(None, fake, fake, 1, fake, 1, None) == kb.KVP_E_INVALID_ARG
