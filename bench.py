#!/usr/bin/env python3
"""Benchmark of the KV-shared attention block on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W]

A step is one pass of the whole path over one batch of synthetic input:
* value: causal prefill / forward of the 8-layer stage share (d_model 2048,
  16 query / 8 KV heads x 128, batch 4, 4096 tokens, layers 5 and 7 share
  layers 4 and 6), in algorithmic TFLOP/s (Q projections of every layer, K/V
  projections of producers, attention over the s(s+1)/2 causal pairs, output
  projections), inputs resident in HBM.
* decode: one new token per sequence through the 32-layer d_model 4096 GQA
  stack (batch 64, 32768-token caches, odd layers share) in tokens/s and
  algorithmic HBM GB/s.
The JSON line also carries the roofline of the dominant kernel (timed with HIP
events on its own stream), the oracle's rate on the host cores, and the
shared-vs-unshared (identity map) ratio.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import kvp_inputs as ki  # noqa: E402

METRIC = "KV-shared prefill attn TFLOP/s + decode tokens/s and HBM GB/s, 1×MI355X"
PEAK_BF16_TFLOPS = 2516.6   # 256 CU x 2.4 GHz x 4096 dense bf16 FLOP/clk
PEAK_HBM_GBS = 8000.0


def log(*a):
    print(*a, file=sys.stderr, flush=True)


# ---------------------------------------------------------------------------
# Algorithmic work
# ---------------------------------------------------------------------------

def prefill_flops(w: ki.Workload, B: int, S: int, tau=None):
    """Per-kind algorithmic FLOPs of one stack forward."""
    tau = w.tau if tau is None else tau
    M = B * S
    nq, nkv = w.a * w.d_h, w.g * w.d_h
    pairs = S * (S + 1) // 2
    out = {"qkv_gemm": 0, "flash_attn": 0, "oproj_gemm": 0}
    for l in range(w.L):
        out["qkv_gemm"] += 2 * M * w.h * nq + (2 * 2 * M * w.h * nkv if tau[l] == l else 0)
        out["flash_attn"] += 4 * B * w.a * w.d_h * pairs
        out["oproj_gemm"] += 2 * M * nq * w.h
    return out


def decode_bytes(w: ki.Workload, lens, tau=None):
    """Per-kind algorithmic HBM bytes of one decode step (bf16)."""
    tau = w.tau if tau is None else tau
    e = 2
    B = len(lens)
    nq, nkv = w.a * w.d_h, w.g * w.d_h
    ctx = int(np.sum(np.asarray(lens, dtype=np.int64) + 1))
    out = {"dec_gemm": 0, "dec_attn": 0, "dec_oproj": 0, "dec_rope": 0}
    for l in range(w.L):
        prod = tau[l] == l
        out["dec_gemm"] += (nq + (2 * nkv if prod else 0)) * w.h * e
        out["dec_oproj"] += w.h * nq * e
        out["dec_attn"] += 2 * ctx * nkv * e                    # K and V of positions [0, len_b]
        out["dec_rope"] += B * (2 * nkv * e if prod else 0)      # appended K, V
    return out


# ---------------------------------------------------------------------------
# Device setup
# ---------------------------------------------------------------------------

class Stack:
    def __init__(self, w: ki.Workload, B: int, max_seq: int, cap: int, fill_npos: int = 0):
        import torch
        from kvp_inputs import device as kd
        from paper_2608_15943_amd import binding as kb
        self.w, self.B, self.cap = w, B, cap
        dt = torch.bfloat16
        self.model = kb.Model(w.L, w.h, w.a, w.g, w.d_h, kb.KVP_DTYPE_BF16, w.tau, max_batch=B,
                              max_seq=max_seq, kv_capacity=cap, rope_base=w.rope_base)
        self.keep = []
        for l in range(w.L):
            prod = w.tau[l] == l
            t = {}
            kinds = [(ki.KIND_WQ, "wq"), (ki.KIND_WO, "wo")]
            if prod:
                kinds += [(ki.KIND_WK, "wk"), (ki.KIND_WV, "wv")]
            for kind, name in kinds:
                rows, cols = ki.weight_shape(w, kind)
                t[name] = torch.empty((rows, cols), dtype=dt, device="cuda")
                kd.fill_weight(w, kind, l, t[name].data_ptr())
            self.model.kvp_set_layer(l, t["wq"].data_ptr(), t["wk"].data_ptr() if prod else 0,
                                     t["wv"].data_ptr() if prod else 0, t["wo"].data_ptr())
            if prod:
                K = torch.empty((B, w.g, cap, w.d_h), dtype=dt, device="cuda")
                V = torch.empty((B, w.g, w.d_h, cap), dtype=dt, device="cuda")
                if fill_npos:
                    kd.fill_cache(w, l, K.data_ptr(), V.data_ptr(), B, cap, fill_npos)
                self.model.kvp_set_kv_slot(l, K.data_ptr(), V.data_ptr())
                t["K"], t["V"] = K, V
            self.keep.append(t)
        torch.cuda.synchronize()


def time_steps(run, model, steps: int, warmup: int):
    """Warm up, then time exactly `steps` calls between two device synchronisations."""
    import torch
    for _ in range(warmup):
        run()
    torch.cuda.synchronize()
    model.kvp_profile_enable(True)
    t0 = time.perf_counter()
    for _ in range(steps):
        run()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    prof = model.kvp_profile_read()
    model.kvp_profile_enable(False)
    return (t1 - t0) * 1e3 / steps, prof


def bench_prefill(w: ki.Workload, steps: int, warmup: int, tau=None):
    import torch
    from kvp_inputs import device as kd
    from paper_2608_15943_amd import binding as kb
    if tau is not None:
        w = w.with_map(tau, "-identity")
    B, S = w.batch, w.seq
    st = Stack(w, B, S, w.kv_capacity)
    x = torch.empty((B, S, w.h), dtype=torch.bfloat16, device="cuda")
    kd.fill_prefill_x(w, x.data_ptr(), B, S)
    y = torch.empty_like(x)
    n = st.model.kvp_workspace_size(kb.KVP_PHASE_PREFILL, B, S)
    ws = torch.empty(n, dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream

    def run():
        st.model.kvp_prefill(x.data_ptr(), y.data_ptr(), B, S, ws.data_ptr(), n, stream)

    ms, prof = time_steps(run, st.model, steps, warmup)
    ok = bool(torch.isfinite(y.float()).all().item())
    del st, x, y, ws
    torch.cuda.empty_cache()
    return ms, prof, ok


def bench_decode(w: ki.Workload, steps: int, warmup: int):
    import torch
    from kvp_inputs import device as kd
    from paper_2608_15943_amd import binding as kb
    lens = w.lengths()
    B = w.batch
    max_len = int(lens.max())
    t0 = time.perf_counter()
    st = Stack(w, B, 1, w.kv_capacity, fill_npos=max_len)
    log(f"[bench] decode setup {time.perf_counter() - t0:.1f}s "
        f"({torch.cuda.memory_allocated() / 2**30:.1f} GiB resident)")
    x = torch.empty((B, w.h), dtype=torch.bfloat16, device="cuda")
    kd.fill_decode_x(w, x.data_ptr(), B)
    y = torch.empty_like(x)
    lens_t = torch.tensor(lens, dtype=torch.int32, device="cuda")
    n = st.model.kvp_workspace_size(kb.KVP_PHASE_DECODE, B)
    ws = torch.empty(n, dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream

    def run():
        st.model.kvp_decode_step(x.data_ptr(), lens_t.data_ptr(), max_len, y.data_ptr(), B,
                                 ws.data_ptr(), n, stream)

    ms, prof = time_steps(run, st.model, steps, warmup)
    ok = bool(torch.isfinite(y.float()).all().item())
    del st, x, y, ws, lens_t
    torch.cuda.empty_cache()
    return ms, prof, ok, lens


# ---------------------------------------------------------------------------
# CPU baseline: the oracle on a bounded sample of the prefill workload
# ---------------------------------------------------------------------------

def cpu_baseline(w: ki.Workload, s_sample: int):
    from oracle import attention as oat
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count() or 1
    ws = []
    for l in range(w.L):
        prod = w.tau[l] == l
        ws.append(oat.LayerWeights(ki.weight(w, ki.KIND_WQ, l),
                                   ki.weight(w, ki.KIND_WK, l) if prod else None,
                                   ki.weight(w, ki.KIND_WV, l) if prod else None,
                                   ki.weight(w, ki.KIND_WO, l)))
    x = ki.prefill_x(w, [0], np.arange(s_sample))[0]
    t0 = time.perf_counter()
    oat.stack_prefill(x, ws, w.tau, w.a, w.g, w.d_h, w.rope_base)
    dt = time.perf_counter() - t0
    flops = sum(prefill_flops(w, 1, s_sample).values())
    return {"value": round(flops / dt / 1e12, 6), "unit": "TFLOP/s", "cores": int(threads),
            "kind": "oracle",
            "sample": f"sequence 0 of 4, first {s_sample} positions (causal prefix, exact), "
                      f"all {w.L} layers, fp64 NumPy; {dt:.1f} s"}


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-decode", action="store_true")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--no-unshared", action="store_true")
    ap.add_argument("--cpu-seq", type=int, default=2048)
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (the KV-shared block is measured on one GPU's share; "
              f"see DESIGN.md for how it shards); --gpus {args.gpus} is not supported", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2608_15943_amd import binding as kb
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    kb.lib()   # fail loudly if the HIP library is missing

    w = ki.stage_share_prefill()
    log(f"[bench] prefill {w.name} steps={args.steps} warmup={args.warmup}")
    ms, prof, finite = bench_prefill(w, args.steps, args.warmup)
    flops = prefill_flops(w, w.batch, w.seq)
    total = sum(flops.values())
    value = total / (ms * 1e-3) / 1e12
    kernels = {k: {"launches": n, "avg_ms": round(t / n, 5)} for k, (n, t) in prof.items()}
    dom = max(("qkv_gemm", "flash_attn", "oproj_gemm"), key=lambda k: prof.get(k, (0, 0.0))[1])
    n_l, t_l = prof[dom]
    per_launch = flops[dom] * args.steps / n_l          # algorithmic FLOPs per launch
    achieved = per_launch / (t_l / n_l * 1e-3) / 1e12
    roofline = {"bound": "mfma", "kernel": dom, "achieved": round(achieved, 2),
                "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / PEAK_BF16_TFLOPS, 4), "traffic": None,
                "flops_per_launch": per_launch, "avg_launch_ms": round(t_l / n_l, 5)}
    log(f"[bench] prefill {ms:.3f} ms/step, {value:.1f} TFLOP/s; kernels {kernels}")

    result = {
        "metric": METRIC, "value": round(value, 2), "unit": "TFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic: seeded SplitMix64 / Irwin-Hall normals, x~N(0,1), W~N(0,0.02), "
                "random-init weights",
        "config": {"workload": w.name, "layers": w.L, "d_model": w.h, "q_heads": w.a,
                   "kv_heads": w.g, "head_dim": w.d_h, "batch": w.batch, "seq_len": w.seq,
                   "causal": True, "map": w.tau, "parallelism": "none (1 GPU)"},
        "roofline": roofline,
        "kernels": kernels,
        "finite": finite,
    }

    if not args.no_unshared:
        ident = list(range(w.L))
        ms_u, _, _ = bench_prefill(w, args.steps, args.warmup, tau=ident)
        ideal = sum(prefill_flops(w, w.batch, w.seq, ident).values()) / total
        result["shared_vs_unshared"] = {"prefill_speedup": round(ms_u / ms, 4),
                                        "prefill_ideal": round(ideal, 4),
                                        "unshared_ms_per_step": round(ms_u, 4)}
        log(f"[bench] identity map {ms_u:.3f} ms/step (speedup {ms_u / ms:.4f}, ideal {ideal:.4f})")

    if not args.no_decode:
        wd = ki.decode_32k()
        log(f"[bench] decode {wd.name}")
        dms, dprof, dfin, lens = bench_decode(wd, max(3, args.steps // 2), max(1, args.warmup // 2))
        db = decode_bytes(wd, lens)
        dtotal = sum(db.values())
        n_a, t_a = dprof["dec_attn"]
        steps_d = max(3, args.steps // 2)
        att_launch = db["dec_attn"] * steps_d / n_a
        att_gbs = att_launch / (t_a / n_a * 1e-3) / 1e9
        result["decode"] = {
            "workload": wd.name, "tokens_per_s": round(wd.batch / (dms * 1e-3), 2),
            "ms_per_step": round(dms, 4), "hbm_gbs": round(dtotal / (dms * 1e-3) / 1e9, 1),
            "hbm_frac": round(dtotal / (dms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
            "bytes_per_step": dtotal, "finite": dfin,
            "roofline": {"bound": "hbm", "kernel": "dec_attn", "achieved": round(att_gbs, 1),
                         "peak": PEAK_HBM_GBS, "unit": "GB/s",
                         "frac": round(att_gbs / PEAK_HBM_GBS, 4), "traffic": None,
                         "bytes_per_launch": att_launch, "avg_launch_ms": round(t_a / n_a, 5)},
            "kernels": {k: {"launches": n, "avg_ms": round(t / n, 5)} for k, (n, t) in dprof.items()},
        }
        log(f"[bench] decode {dms:.3f} ms/step, {wd.batch / (dms * 1e-3):.1f} tok/s, "
            f"attention {att_gbs:.0f} GB/s")

    if not args.no_cpu:
        log(f"[bench] oracle CPU baseline (first {args.cpu_seq} positions of one sequence)")
        result["cpu_baseline"] = cpu_baseline(w, args.cpu_seq)

    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
