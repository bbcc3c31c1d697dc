"""The benchmark's algorithmic FLOPs (the numerator of its headline TFLOP/s) against the
oracle's App. A.7 layer model: the same projections, and causal attention over
S (S + 1) / 2 query-key pairs (diagonal included) where the paper's model takes S^2 / 2,
so the two differ by exactly 2 B a d_h S per layer."""
import bench
import kvp_inputs as ki
from oracle import planner as opl


def _oracle_total(w, B, S, tau):
    tot = 0
    for l in range(w.L):
        f0, f1 = opl.layer_flops_prefill(B, S, w.h, w.a, w.g, causal=True)
        tot += f0 if tau[l] == l else f1
    return tot


def test_prefill_flops_match_the_paper_model():
    for w in (ki.stage_share_prefill(), ki.stage_70b_prefill([0] * 10)):
        B, S = w.batch, w.seq
        for tau in (w.tau, list(range(w.L))):
            got = sum(bench.prefill_flops(w, B, S, tau).values())
            assert got - _oracle_total(w, B, S, tau) == w.L * 2 * B * w.a * w.d_h * S


def test_backward_flops_are_twice_the_forward():
    w = ki.stage_share_prefill()
    f = bench.prefill_flops(w, w.batch, w.seq)
    b = bench.backward_flops(w, w.batch, w.seq)
    assert b["bwd_gemm"] == 2 * (f["qkv_gemm"] + f["oproj_gemm"])
    assert b["bwd_attn_algorithmic"] == 2 * f["flash_attn"]


def test_decode_bytes_count_every_cached_position_once():
    w = ki.decode_32k()
    lens = w.lengths()
    db = bench.decode_bytes(w, lens)
    ctx = int(sum(int(n) + 1 for n in lens))
    assert db["dec_attn"] == w.L * 2 * ctx * w.g * w.d_h * 2
