"""FIR comparison of the placement strategies (Sec. 2.7, Table 2; App. A.1, Tables A1-A3).

For a dense decoder split evenly over P pipeline stages, with the LM head on
the last stage, this prints the FLOP Imbalance Ratio of the baseline and of
the three placement archetypes of Sec. 2.5 under the same budget of k
KV-sharing layers: Uniform and Symmetric Bipolar (kvp_place) and
Architecture-Balanced (Algorithm 1, kvp_plan_fir with m = k).  Every number
comes from the C++ planner in libkvpipe.so; this module only builds the
inputs (per-layer FLOPs from kvp_layer_flops, the LM head as 2 b s h V) and
formats the result.

    python -m paper_2608_15943_amd.fir_table --pp 8 --seq 8192 --k 4

The defaults are the LLaMA2-7B shape (32 layers, h = 4096, 32 heads, MHA,
SwiGLU width 11008, vocabulary 32000, micro-batch 1) with causal score and
context FLOPs, the setting of Table 2.
"""
from __future__ import annotations

import argparse
import json
import sys

from . import binding as kb

STRATEGIES = ("baseline", "uniform", "symmetric_bipolar", "arch_balanced")


def fir_table(L=32, P=8, b=1, s=8192, h=4096, a=32, g=32, ffn=11008, vocab=32000, k=4,
              eps=0.02, causal=True, admissible=None, alpha=-1.0):
    """Rows {strategy, layers (1-indexed), stage_flops, fir} for one configuration."""
    if L < 1 or P < 1 or P > L:
        raise ValueError("need 1 <= P <= L")
    stage = [l * P // L for l in range(L)]
    f0, f1 = kb.kvp_layer_flops(b, s, h, a, g, ffn=ffn, causal=causal)
    ff, fs = [f0] * L, [f1] * L
    lm = 2.0 * b * s * h * vocab
    rows = []
    for name in STRATEGIES:
        if name == "baseline":
            z = [0] * L
        elif name == "uniform":
            z = kb.kvp_place(kb.KVP_PLACE_UNIFORM, stage, k, admissible, alpha, P=P)[0]
        elif name == "symmetric_bipolar":
            z = kb.kvp_place(kb.KVP_PLACE_SYMMETRIC_BIPOLAR, stage, k, admissible, alpha, P=P)[0]
        else:
            z = kb.kvp_plan_fir(stage, ff, fs, lm, eps, m=k, admissible=admissible, alpha=alpha,
                                P=P)["z"]
        F = kb.kvp_stage_flops(stage, ff, fs, z, lm, P=P)
        rows.append(dict(strategy=name, layers=[l + 1 for l in range(L) if z[l]], stage_flops=F,
                         fir=kb.kvp_fir(F)))
    return rows


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--layers", type=int, default=32)
    ap.add_argument("--pp", type=int, default=8)
    ap.add_argument("--mbs", type=int, default=1)
    ap.add_argument("--seq", type=int, default=8192)
    ap.add_argument("--hidden", type=int, default=4096)
    ap.add_argument("--heads", type=int, default=32)
    ap.add_argument("--kv-heads", type=int, default=None, help="default: --heads (MHA)")
    ap.add_argument("--ffn", type=int, default=11008)
    ap.add_argument("--vocab", type=int, default=32000)
    ap.add_argument("--k", type=int, default=4, help="KV-sharing layers (budget m)")
    ap.add_argument("--eps", type=float, default=0.02)
    ap.add_argument("--alpha", type=float, default=-1.0, help="App. A.3 guardrail (< 0: off)")
    ap.add_argument("--full-s2", action="store_true", help="score/context over s^2 pairs")
    ap.add_argument("--json", action="store_true")
    args = ap.parse_args(argv)
    rows = fir_table(L=args.layers, P=args.pp, b=args.mbs, s=args.seq, h=args.hidden, a=args.heads,
                     g=args.kv_heads or args.heads, ffn=args.ffn, vocab=args.vocab, k=args.k,
                     eps=args.eps, causal=not args.full_s2, alpha=args.alpha)
    if args.json:
        print(json.dumps(rows))
        return 0
    print(f"{'strategy':<18} {'FIR':>12}  layers (1-indexed)")
    for r in rows:
        print(f"{r['strategy']:<18} {r['fir']:>12.9f}  {','.join(map(str, r['layers'])) or '-'}")
    print()
    print(f"{'stage FLOPs':<18} " + " ".join(f"{i:>9}" for i in range(args.pp)))
    for r in rows:
        print(f"{r['strategy']:<18} " + " ".join(f"{v:9.3E}" for v in r["stage_flops"]))
    return 0


if __name__ == "__main__":
    sys.exit(main())
