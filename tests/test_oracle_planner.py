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
