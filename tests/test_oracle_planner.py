"""Pins for the planner oracle: the paper's printed tables, hand-computed toys,
closed forms of App. A.7, and the edge cases of Algorithm 1."""
import math
import os

import pytest

from oracle import planner as pl

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paper_fir_tables.txt")


def golden():
    vals = {}
    with open(GOLDEN) as f:
        for line in f:
            if not line.strip() or line.startswith("#"):
                continue
            key, val = line.split()[:2]
            vals[key] = val
    return vals


# LLaMA2-7B public shape (not printed in the paper): h=4096, 32 heads (MHA),
# SwiGLU width 11008, vocab 32000.  MBS = 1.
H, A, FFN, VOCAB, L = 4096, 32, 11008, 32000, 32


def llama2_7b(S, P):
    f0, f1 = pl.layer_flops_prefill(1, S, H, A, A, ffn=FFN, causal=True)
    stage = [l * P // L for l in range(L)]
    lm = pl.mm_flops(S, H, VOCAB)
    return stage, [f0] * L, [f1] * L, lm


def test_table1_stage_flops_and_table2_baseline_fir():
    g = golden()
    stage, ff, fs, lm = llama2_7b(8192, 8)
    F = pl.stage_flops(stage, 8, ff, fs, [0] * L, lm)
    # Table 1 prints three significant digits for the body stages.
    assert f"{F[0]:.2E}" == g["table1_stage_flops_body"]
    # Table 2 prints ten digits; the causal-half reading reproduces all of them.
    assert abs(pl.fir(F) - float(g["table2_fir_baseline"])) < 1e-9
    # The printed tail (1.763E+13) is ~0.12 % above the value that gives the printed FIR.
    assert abs(F[7] / float(g["table1_stage_flops_tail"]) - 1) < 2e-3


def test_full_s2_reading_does_not_reproduce_table2():
    # The alternative reading (full s^2 score/context FLOPs) misses Table 2 by far.
    f0, f1 = pl.layer_flops_prefill(1, 8192, H, A, A, ffn=FFN, causal=False)
    stage = [l // 4 for l in range(L)]
    F = pl.stage_flops(stage, 8, [f0] * L, [f1] * L, [0] * L, pl.mm_flops(8192, H, VOCAB))
    assert abs(pl.fir(F) - 1.119453925) > 1e-3


def test_table3_baseline_firs():
    g = golden()
    stage, ff, fs, lm = llama2_7b(4096, 2)
    assert abs(pl.fir(pl.stage_flops(stage, 2, ff, fs, [0] * L, lm))
               - float(g["table3_fir_pp2_s4k_baseline"])) < 2e-4
    stage, ff, fs, lm = llama2_7b(8192, 4)
    assert abs(pl.fir(pl.stage_flops(stage, 4, ff, fs, [0] * L, lm))
               - float(g["table3_fir_pp4_s8k_baseline"])) < 5e-4


def test_algorithm1_arch_balanced_llama2_pp8():
    g = golden()
    stage, ff, fs, lm = llama2_7b(8192, 8)
    res = pl.plan_fir(stage, 8, ff, fs, lm, eps=0.02, m=4)
    conv = [l + 1 for l in range(L) if res.z[l]]
    assert conv == [int(x) for x in g["layers_arch_balanced"].split(",")]
    assert res.n_converted == 4 and res.stop_reason == pl.STOP_FIR_MET
    # With eps below the last step the budget m = 4 is what stops it.
    res_b = pl.plan_fir(stage, 8, ff, fs, lm, eps=1e-4, m=4)
    assert res_b.z == res.z and res_b.stop_reason == pl.STOP_BUDGET
    assert abs(res.fir - float(g["table2_fir_arch_balanced"])) < 2e-5
    assert abs(res.fir - float(g["table3_fir_pp8_s8k_kvpipe"])) < 1e-4
    assert abs(res.stage_flops[7] / float(g["tableA3_arch_stage_flops_tail"]) - 1) < 2e-3
    # FIR falls monotonically along the tail conversions.
    assert all(b < a for a, b in zip(res.fir_trace, res.fir_trace[1:]))


def test_uniform_and_symmetric_placements_tables_a1_a2_and_table2():
    g = golden()
    stage, ff, fs, lm = llama2_7b(8192, 8)
    # Uniform: the layer set printed in the sensitivity table.
    z = [0] * L
    for l in (int(x) for x in g["layers_uniform"].split(",")):
        z[l - 1] = 1
    F = pl.stage_flops(stage, 8, ff, fs, z, lm)
    assert f"{F[4]:.2E}" == g["tableA1_uniform_stage_flops_shared1"]
    assert abs(F[7] / float(g["tableA1_uniform_stage_flops_tail"]) - 1) < 2e-3
    assert abs(pl.fir(F) - float(g["table2_fir_uniform"])) < 4e-5
    # Symmetric bipolar as Table A2 lays it out: two shared layers in stages 3 and 7
    # (the tail-most layers of each).
    z = [0] * L
    for l in (15, 16, 31, 32):
        z[l - 1] = 1
    F = pl.stage_flops(stage, 8, ff, fs, z, lm)
    assert f"{F[3]:.2E}" == g["tableA2_symmetric_stage_flops_shared2"]
    assert abs(F[7] / float(g["tableA2_symmetric_stage_flops_tail"]) - 1) < 2e-3
    assert abs(pl.fir(F) - float(g["table2_fir_symmetric"])) < 4e-5


def per_stage(stage, z, P):
    c = [0] * P
    for l, zl in enumerate(z):
        c[stage[l]] += zl
    return c


def test_uniform_rule_reproduces_printed_layers_and_table_a1():
    g = golden()
    stage, ff, fs, lm = llama2_7b(8192, 8)
    z, n, stop = pl.place_uniform(stage, 8, 4)
    assert [l + 1 for l in range(L) if z[l]] == [int(x) for x in g["layers_uniform"].split(",")]
    assert per_stage(stage, z, 8) == [int(x) for x in g["tableA1_uniform_shared_per_stage"].split(",")]
    assert n == 4 and stop == pl.STOP_BUDGET
    F = pl.stage_flops(stage, 8, ff, fs, z, lm)
    assert f"{F[5]:.2E}" == g["tableA1_uniform_stage_flops_shared1"]
    assert abs(pl.fir(F) - float(g["table2_fir_uniform"])) < 4e-5


def test_symmetric_rule_reproduces_table_a2():
    g = golden()
    stage, ff, fs, lm = llama2_7b(8192, 8)
    z, n, stop = pl.place_symmetric_bipolar(stage, 8, 4)
    assert per_stage(stage, z, 8) == [int(x) for x in g["tableA2_symmetric_shared_per_stage"].split(",")]
    assert [l + 1 for l in range(L) if z[l]] == [15, 16, 31, 32]      # tail-most of stages 3, 7
    assert n == 4 and stop == pl.STOP_BUDGET
    F = pl.stage_flops(stage, 8, ff, fs, z, lm)
    assert abs(pl.fir(F) - float(g["table2_fir_symmetric"])) < 4e-5
    # The sensitivity table's layer set (stages 4 and 7) has the same stage-FLOPs
    # multiset, so the two printed descriptions agree on the FIR.
    z2 = [0] * L
    for l in (int(x) for x in g["layers_symmetric_sensitivity"].split(",")):
        z2[l - 1] = 1
    F2 = pl.stage_flops(stage, 8, ff, fs, z2, lm)
    assert sorted(F2) == sorted(F)
    assert abs(pl.fir(F2) - pl.fir(F)) < 1e-15


def test_strategy_table_reproduces_table2_and_table_a3():
    g = golden()
    stage, ff, fs, lm = llama2_7b(8192, 8)
    rows = {name: (z, F, f) for name, z, F, f in pl.strategy_table(stage, 8, ff, fs, lm, k=4, eps=1e-4)}
    assert abs(rows["baseline"][2] - float(g["table2_fir_baseline"])) < 1e-9
    assert abs(rows["uniform"][2] - float(g["table2_fir_uniform"])) < 4e-5
    assert abs(rows["symmetric_bipolar"][2] - float(g["table2_fir_symmetric"])) < 4e-5
    assert abs(rows["arch_balanced"][2] - float(g["table2_fir_arch_balanced"])) < 2e-5
    assert per_stage(stage, rows["arch_balanced"][0], 8) == [
        int(x) for x in g["tableA3_arch_shared_per_stage"].split(",")]
    # The paper's ranking: each archetype closer to 1 than the one before.
    f = [rows[k][2] for k in ("baseline", "uniform", "symmetric_bipolar", "arch_balanced")]
    assert f == sorted(f, reverse=True)
    # Same budget, same total FLOPs removed: only where they are removed differs.
    tot = {k: sum(v[1]) for k, v in rows.items()}
    assert len({tot["uniform"], tot["symmetric_bipolar"], tot["arch_balanced"]}) == 1


# Toy partition for the placements: 12 layers, stages {0-2},{3-5},{6-8},{9-11}.
def test_uniform_toys():
    T = [l // 3 for l in range(12)]
    on = lambda z: [l for l in range(len(z)) if z[l]]
    # k = 2: span = stages 2-3 = layers 6..11, targets 11 and 11 - round(5) = 6.
    assert on(pl.place_uniform(T, 4, 2)[0]) == [6, 11]
    # k = 4: span = all, targets 11, 11 - round(11/3) = 7, 11 - round(22/3) = 4, 0;
    # layer 0 is never converted, so its target moves right to layer 1.
    assert on(pl.place_uniform(T, 4, 4)[0]) == [1, 4, 7, 11]
    # k = 1: the last layer; k = 0: nothing.
    assert on(pl.place_uniform(T, 4, 1)[0]) == [11]
    assert pl.place_uniform(T, 4, 0) == ([0] * 12, 0, pl.STOP_BUDGET)
    # More than the 11 convertible layers: all of them, then stop.
    z, n, stop = pl.place_uniform(T, 4, 12)
    assert on(z) == list(range(1, 12)) and n == 11 and stop == pl.STOP_NO_CONVERTIBLE
    # Guardrail alpha = 0.5: 1-indexed layers >= 6 (0-indexed >= 5).  Targets 11, 7, 4, 0:
    # 4 and 0 have no free layer on their left and move right to 5 and 6.
    assert on(pl.place_uniform(T, 4, 4, alpha=0.5)[0]) == [5, 6, 7, 11]
    # One stage: span = all five layers, targets 4 and 0 -> 1.
    assert on(pl.place_uniform([0] * 5, 1, 2)[0]) == [1, 4]


def test_symmetric_toys():
    T = [l // 3 for l in range(12)]
    on = lambda z: [l for l in range(len(z)) if z[l]]
    # Anchors: layer 11 (last stage) and layer 5 (last of stage (4 - 1) // 2 = 1).
    assert on(pl.place_symmetric_bipolar(T, 4, 1)[0]) == [11]
    assert on(pl.place_symmetric_bipolar(T, 4, 3)[0]) == [5, 10, 11]
    assert on(pl.place_symmetric_bipolar(T, 4, 7)[0]) == [3, 4, 5, 8, 9, 10, 11]
    # Guardrail alpha = 0.5 (0-indexed >= 5): after 11, 5, 10 the middle anchor has
    # nothing left and hands its turn to the last one (9).
    assert on(pl.place_symmetric_bipolar(T, 4, 4, alpha=0.5)[0]) == [5, 9, 10, 11]
    # The last anchor walks into the middle anchor's layers without taking one twice.
    z, n, stop = pl.place_symmetric_bipolar(T, 4, 12)
    assert on(z) == list(range(1, 12)) and n == 11 and stop == pl.STOP_NO_CONVERTIBLE
    # P = 2: the middle stage is stage 0 (anchor 5); P = 1: one anchor.
    assert on(pl.place_symmetric_bipolar([l // 6 for l in range(12)], 2, 2)[0]) == [5, 11]
    assert [l for l, x in enumerate(pl.place_symmetric_bipolar([0] * 5, 1, 2)[0]) if x] == [3, 4]


def test_placement_invariants_brute_force():
    import random
    rng = random.Random(5)
    for _ in range(300):
        P = rng.randint(1, 8)
        N = rng.randint(2, 6)
        Lr = P * N
        stage = [l // N for l in range(Lr)]
        # Equal stages, k <= P: one conversion in each of the last k stages.
        k = rng.randint(0, P)
        z, n, stop = pl.place_uniform(stage, P, k)
        assert per_stage(stage, z, P) == [0] * (P - k) + [1] * k
        # Symmetric, k small enough to stay inside the anchor stages: ceil(k/2) at the
        # tail of the last stage, floor(k/2) at the tail of the middle stage.
        if P >= 2:
            mid = (P - 1) // 2
            cap = N - 1 if mid == 0 else N
            k2 = rng.randint(0, 2 * min(N, cap))
            z, n, stop = pl.place_symmetric_bipolar(stage, P, k2)
            c = per_stage(stage, z, P)
            assert c[P - 1] == (k2 + 1) // 2 and c[mid] == k2 // 2 and sum(c) == k2
            for i in (P - 1, mid):
                got = [l for l in range(Lr) if z[l] and stage[l] == i]
                end = max(l for l in range(Lr) if stage[l] == i)
                assert got == list(range(end - len(got) + 1, end + 1))
        # Any partition, mask and k: both place min(k, free layers), never layer 0,
        # never an inadmissible layer.
        cuts = sorted(rng.sample(range(1, Lr), P - 1)) if P > 1 else []
        stage = [sum(1 for c in cuts if l >= c) for l in range(Lr)]
        adm = [rng.random() < 0.7 for _ in range(Lr)]
        k = rng.randint(0, Lr + 2)
        free = sum(adm[1:])
        for fn in (pl.place_uniform, pl.place_symmetric_bipolar):
            z, n, stop = fn(stage, P, k, admissible=adm)
            assert n == sum(z) == min(k, free) and z[0] == 0
            assert all(adm[l] for l in range(Lr) if z[l])
            assert stop == (pl.STOP_BUDGET if k <= free else pl.STOP_NO_CONVERTIBLE)


def test_placement_rejects_bad_partitions():
    with pytest.raises(ValueError):
        pl.place_uniform([0, 1, 0], 2, 1)
    with pytest.raises(ValueError):
        pl.place_symmetric_bipolar([0, 2, 2], 3, 1)
    with pytest.raises(ValueError):
        pl.place_uniform([0, 0, 1], 2, -1)


# ---------------------------------------------------------------------------
# Hand-computed toys: stages {0,1,2},{3,4,5},{6,7,8},{9,10,11}, F(0) = 10, eps = 0.01.
# ---------------------------------------------------------------------------
TOY_STAGE = [l // 3 for l in range(12)]


def test_toy_t1_tail_only():
    res = pl.plan_fir(TOY_STAGE, 4, [10] * 12, [7] * 12, 6, eps=0.01)
    # F = [30,30,30,36] -> FIR 36/31.5; convert 11 -> 33/30.75; convert 10 -> 1.0.
    assert res.z == [0] * 10 + [1, 1]
    assert res.stage_flops == [30, 30, 30, 30]
    assert res.fir == 1.0 and res.stop_reason == pl.STOP_FIR_MET
    assert abs(res.fir_trace[0] - 36 / 31.5) < 1e-15
    assert abs(res.fir_trace[1] - 33 / 30.75) < 1e-15
    assert pl.map_from_mask(res.z) == list(range(10)) + [9, 9]


def test_toy_t2_whole_tail_stage():
    res = pl.plan_fir(TOY_STAGE, 4, [10] * 12, [7] * 12, 9, eps=0.01)
    # F = [30,30,30,39] -> convert 11, 10, 9 -> [30,30,30,30]
    assert [l for l in range(12) if res.z[l]] == [9, 10, 11]
    assert res.fir == 1.0
    assert pl.map_from_mask(res.z)[9:] == [8, 8, 8]      # producer on the previous stage
    assert abs(res.fir_trace[0] - 39 / 32.25) < 1e-15


def test_toy_t3_retarget_and_tie_break():
    res = pl.plan_fir(TOY_STAGE, 4, [10] * 12, [4] * 12, 4, eps=0.01, m=3)
    # Convert 11: F=[30,30,30,28], avg 29.5, tail <= 1.01*29.5 so take the argmax;
    # stages 0-2 tie and the tail-most (2) wins -> convert 8; then 0,1 tie -> stage 1 -> 5.
    assert [l for l in range(12) if res.z[l]] == [5, 8, 11]
    assert res.stop_reason == pl.STOP_BUDGET
    assert res.stage_flops == [30, 24, 24, 28]
    assert abs(res.fir - 30 / 26.5) < 1e-15
    assert abs(res.fir_trace[1] - 30 / 29.5) < 1e-15
    # The final state is returned even though it is worse than the start.
    assert res.fir > res.fir_trace[0]
    tau = pl.map_from_mask(res.z)
    assert (tau[5], tau[8], tau[11]) == (4, 7, 10)


def test_stop_no_convertible_and_guardrail():
    # Admissible only layer 11: after converting it the tail is still heavy -> break.
    adm = [False] * 11 + [True]
    res = pl.plan_fir(TOY_STAGE, 4, [10] * 12, [9] * 12, 30, eps=0.01, admissible=adm)
    assert res.z == [0] * 11 + [1] and res.stop_reason == pl.STOP_NO_CONVERTIBLE
    # Guardrail C_alpha with alpha = 0.5, L = 32: 1-indexed layers >= 16 admissible.
    ca = pl.guardrail_admissible(32, 0.5)
    assert ca.index(True) == 15 and all(ca[15:])
    # Layer 0 is never converted, even when it is the only candidate left.
    # Stage 0 = {0, 1} is the bottleneck; after layer 1 only layer 0 is left.
    res = pl.plan_fir([0, 0, 1], 2, [100, 100, 10], [99, 99, 9], 0, eps=0.01)
    assert res.z == [0, 1, 0] and res.stop_reason == pl.STOP_NO_CONVERTIBLE


def test_budget_and_tolerance_edges():
    stage, ff, fs, lm = llama2_7b(8192, 8)
    res = pl.plan_fir(stage, 8, ff, fs, lm, eps=1.0)
    assert sum(res.z) == 0 and res.stop_reason == pl.STOP_FIR_MET
    res = pl.plan_fir(stage, 8, ff, fs, lm, eps=1e-9, m=0)   # m <= 0 means m = L
    assert res.n_converted <= L


def test_closed_forms_app_a7():
    h, s, b = 4096, 8192, 2
    # Eq. (qkv_mha): MHA projections are 6bsh^2; Eq. (qkv_gqa) for r = 4.
    f0, f1 = pl.layer_flops_prefill(b, s, h, 32, 32, causal=False)
    assert f0 == 8 * b * s * h * h + 4 * b * s * s * h          # Eq. (attn_mha_total)
    assert f0 - f1 == 4 * b * s * h * h
    f0, f1 = pl.layer_flops_prefill(b, s, h, 32, 8, causal=False)
    assert f0 == 4 * b * s * h * h + 4 * b * s * h * h // 4 + 4 * b * s * s * h   # Eq. (attn_gqa_total)
    # Per-token forms, Eqs. (attn_mha_token) and (attn_gqa_token).
    assert pl.per_token_attn_flops(h, s, 1) == 8 * h * h + 4 * s * h
    assert f0 / (b * s) == pl.per_token_attn_flops(h, s, 4)
    # Eqs. (gqa_skv_flop_saving), (gqa_skv_cache_saving).
    dF, dB = pl.gqa_sharing_savings(h, 4, 2)
    assert dF == 4 * h * h / 4 and dB == 2 * (h / 4) * 2
    assert (f0 - f1) / (b * s) == dF
    # Decode: one token against ctx keys.
    f0, f1 = pl.layer_flops_decode(64, 32768, 4096, 32, 8)
    assert f0 == 64 * pl.per_token_attn_flops(4096, 32768, 4)


def test_map_from_mask_and_canonicalize():
    # The sharing maps of the workloads: tail-first pairs, alternate layers, groups of four.
    assert pl.map_from_mask([0, 1, 0, 1]) == [0, 0, 2, 2]
    assert pl.map_from_mask([0, 0, 0, 0, 0, 1, 0, 1]) == [0, 1, 2, 3, 4, 4, 6, 6]
    assert pl.map_from_mask([0, 1, 1, 1] * 2) == [0, 0, 0, 0, 4, 4, 4, 4]
    with pytest.raises(ValueError):
        pl.map_from_mask([1, 0])
    # Chains resolve to the root producer; forward references are rejected.
    assert pl.canonicalize_map([0, 0, 1, 2, 4]) == [0, 0, 0, 0, 4]
    with pytest.raises(ValueError):
        pl.canonicalize_map([0, 2, 2])
    with pytest.raises(ValueError):
        pl.canonicalize_map([1])


def test_70b_stage_map_from_fir_rule():
    """The 70B-shaped stage: 80 layers on 8 stages, stage tail 30 % heavier.

    Each conversion removes 4bsh^2/r, ~7.7 % of one layer, far less than the
    30 % excess, so the rule empties the tail stage of admissible layers
    (all but its first) and stops: the stage keeps 1 producer and 9 consumers.
    """
    Lw, P = 80, 8
    f0, f1 = pl.layer_flops_prefill(1, 8192, 8192, 64, 8, causal=True)
    assert 0.07 < (f0 - f1) / f0 < 0.08
    stage = [l // 10 for l in range(Lw)]
    adm = [l % 10 != 0 for l in range(Lw)]
    lm = 0.3 * 10 * f0
    res = pl.plan_fir(stage, P, [f0] * Lw, [f1] * Lw, lm, eps=0.05, admissible=adm)
    assert [l for l in range(Lw) if res.z[l]] == list(range(71, 80))
    assert res.stop_reason == pl.STOP_NO_CONVERTIBLE
    tau = pl.map_from_mask(res.z)
    assert [t - 70 for t in tau[70:]] == [0] * 10
    assert res.fir_trace[0] > res.fir > 1.05
