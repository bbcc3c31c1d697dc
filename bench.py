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
* train: forward with saved activations plus the backward of the same 8-layer
  stage (dX and every weight gradient), in TFLOP/s of 3x the forward's FLOPs.
The JSON line also carries the roofline of the dominant kernel (timed with HIP
events on its own stream) against the datasheet peak and against the peak this
device measurably delivers (a bf16 matrix-core loop and a streaming read, run
first), the oracle's rate on the host cores, and the shared-vs-unshared
(identity map) ratio.
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


def backward_flops(w: ki.Workload, B: int, S: int, tau=None):
    """Per-kind FLOPs of one stack backward.  Algorithmic: the projection gradients (dO, dW_O,
    dW_QKV, dX: twice the forward projections) and the four attention products (dV, dP, dQ, dK:
    twice the forward attention).  Executed by the attention kernels, over the causal pairs:
    the dK/dV kernel recomputes S and runs dP, dV, dK (4 products), the dQ kernel recomputes S
    and dP and runs dQ (3)."""
    tau = w.tau if tau is None else tau
    M = B * S
    nq, nkv = w.a * w.d_h, w.g * w.d_h
    unit = 2 * B * w.a * w.d_h * (S * (S + 1) // 2)     # one causal [S x S x d] product, all heads
    gemm = 0
    for l in range(w.L):
        npj = nq + (2 * nkv if tau[l] == l else 0)
        gemm += 2 * M * w.h * nq * 2 + 2 * M * w.h * npj * 2
    return {"bwd_gemm": gemm, "bwd_attn_algorithmic": 4 * unit * w.L,
            "bwd_attn_kv_executed": 4 * unit * w.L, "bwd_attn_q_executed": 3 * unit * w.L}


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
    """Weights and KV slots of a workload on the device.  alias_of maps a producer to an
    earlier producer whose slot memory it reuses (used only when the unshared map does
    not fit in HBM; timing is unaffected because every slot is far larger than the caches)."""

    def __init__(self, w: ki.Workload, B: int, max_seq: int, cap: int, fill_npos: int = 0,
                 alias_of=None, slots: bool = True):
        import torch
        from kvp_inputs import device as kd
        from paper_2608_15943_amd import binding as kb
        self.w, self.B, self.cap = w, B, cap
        dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
        self.model = kb.Model(w.L, w.h, w.a, w.g, w.d_h,
                              kb.KVP_DTYPE_BF16 if w.dtype == "bf16" else kb.KVP_DTYPE_FP32, w.tau,
                              max_batch=B, max_seq=max_seq, kv_capacity=cap, rope_base=w.rope_base)
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
            if prod and slots:
                if alias_of and l in alias_of:
                    K, V = self.keep[alias_of[l]]["K"], self.keep[alias_of[l]]["V"]
                else:
                    K = torch.empty((B, w.g, cap, w.d_h), dtype=dt, device="cuda")
                    V = torch.empty((B, w.g, w.d_h, cap), dtype=dt, device="cuda")
                    if fill_npos:
                        kd.fill_cache(w, l, K.data_ptr(), V.data_ptr(), B, cap, fill_npos)
                self.model.kvp_set_kv_slot(l, K.data_ptr(), V.data_ptr())
                t["K"], t["V"] = K, V
            self.keep.append(t)
        torch.cuda.synchronize()


LAST_STEP_MS = []   # per-step times (ms) of the last time_steps call


def time_steps(run, model, steps: int, warmup: int):
    """Warm up, time exactly `steps` calls between two device synchronisations, then time
    another `steps` calls with the library's per-launch HIP events on (for the per-kernel
    figures), so that the step time itself is not perturbed by the event records.  The timed
    calls are also separated by events on the launch stream (one record between calls), whose
    per-step times are kept in LAST_STEP_MS for the spread of the step time."""
    import torch
    for _ in range(warmup):
        run()
    torch.cuda.synchronize()
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    t0 = time.perf_counter()
    evs[0].record()
    for i in range(steps):
        run()
        evs[i + 1].record()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    LAST_STEP_MS[:] = [evs[i].elapsed_time(evs[i + 1]) for i in range(steps)]
    model.kvp_profile_enable(True)
    for _ in range(steps):
        run()
    torch.cuda.synchronize()
    prof = model.kvp_profile_read()
    model.kvp_profile_enable(False)
    return (t1 - t0) * 1e3 / steps, prof


def step_spread():
    """Min / median / max of the per-step times of the last time_steps call (ms)."""
    t = sorted(LAST_STEP_MS)
    if not t:
        return None
    return {"min": round(t[0], 4), "median": round(t[len(t) // 2], 4), "max": round(t[-1], 4)}


def bench_prefill(w: ki.Workload, steps: int, warmup: int, tau=None):
    import torch
    from kvp_inputs import device as kd
    from paper_2608_15943_amd import binding as kb
    if tau is not None:
        w = w.with_map(tau, "-identity")
    B, S = w.batch, w.seq
    st = Stack(w, B, S, w.kv_capacity)
    x = torch.empty((B, S, w.h), dtype=torch.bfloat16 if w.dtype == "bf16" else torch.float32,
                    device="cuda")
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


def bench_train(w: ki.Workload, steps: int, warmup: int):
    """One training step of the stack: kvp_train_forward (the prefill kernels, keeping Q, O, the
    layer inputs and the log-sum-exp) then kvp_backward (dX and every weight gradient, fp32)."""
    import torch
    from kvp_inputs import device as kd
    from paper_2608_15943_amd import binding as kb
    B, S = w.batch, w.seq
    st = Stack(w, B, S, w.kv_capacity)
    m = st.model
    x = torch.empty((B, S, w.h), dtype=torch.bfloat16, device="cuda")
    kd.fill_prefill_x(w, x.data_ptr(), B, S)
    y = torch.empty_like(x)
    dy = torch.empty((B, S, w.h), dtype=torch.float32, device="cuda")
    kd.fill_prefill_dy(w, dy.data_ptr(), B, S)
    dx = torch.empty_like(dy)
    grads = []
    for l in range(w.L):
        prod = w.tau[l] == l
        g = {"q": torch.empty((w.a * w.d_h, w.h), device="cuda"),
             "o": torch.empty((w.h, w.a * w.d_h), device="cuda")}
        if prod:
            g["k"] = torch.empty((w.g * w.d_h, w.h), device="cuda")
            g["v"] = torch.empty((w.g * w.d_h, w.h), device="cuda")
        m.kvp_set_layer_grads(l, g["q"].data_ptr(), g["k"].data_ptr() if prod else 0,
                              g["v"].data_ptr() if prod else 0, g["o"].data_ptr())
        grads.append(g)
    nf = m.kvp_workspace_size(kb.KVP_PHASE_PREFILL, B, S)
    nb = m.kvp_workspace_size(kb.KVP_PHASE_BACKWARD, B, S)
    ns = m.kvp_train_saved_size(B, S)
    ws = torch.empty(max(nf, nb), dtype=torch.uint8, device="cuda")
    saved = torch.empty(ns, dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    log(f"[bench] train {w.name}: saved {ns / 2**30:.2f} GiB, backward workspace {nb / 2**30:.2f} GiB")

    def run():
        m.kvp_train_forward(x.data_ptr(), y.data_ptr(), B, S, saved.data_ptr(), ns, ws.data_ptr(), nf,
                            stream)
        m.kvp_backward(x.data_ptr(), dy.data_ptr(), dx.data_ptr(), B, S, saved.data_ptr(), ns,
                       ws.data_ptr(), nb, stream)

    ms, prof = time_steps(run, m, steps, warmup)
    ok = bool(torch.isfinite(dx).all().item()) and all(
        bool(torch.isfinite(t).all().item()) for g in grads for t in g.values())
    del st, x, y, dy, dx, grads, ws, saved
    torch.cuda.empty_cache()
    return ms, prof, ok


def train_entry(w: ki.Workload, steps: int, warmup: int):
    ms, prof, ok = bench_train(w, steps, warmup)
    ff = prefill_flops(w, w.batch, w.seq)
    bf = backward_flops(w, w.batch, w.seq)
    fwd_flops = sum(ff.values())
    algo = fwd_flops + bf["bwd_gemm"] + bf["bwd_attn_algorithmic"]     # = 3 x forward
    kern = {k: {"launches": n, "avg_ms": round(t / n, 5)} for k, (n, t) in prof.items()}
    tot = {k: t / steps for k, (n, t) in prof.items()}                # ms per step per kind
    bwd_ms = sum(v for k, v in tot.items() if k.startswith("bwd_"))
    rates = {
        "bwd_attn_kv": round(bf["bwd_attn_kv_executed"] / (tot["bwd_attn_kv"] * 1e-3) / 1e12, 1),
        "bwd_attn_q": round(bf["bwd_attn_q_executed"] / (tot["bwd_attn_q"] * 1e-3) / 1e12, 1),
        "bwd_attn_algorithmic": round(bf["bwd_attn_algorithmic"] /
                                      ((tot["bwd_attn_kv"] + tot["bwd_attn_q"]) * 1e-3) / 1e12, 1),
        "bwd_gemm": round(bf["bwd_gemm"] / (tot["bwd_gemm"] * 1e-3) / 1e12, 1),
    }
    out = {"workload": w.name, "ms_per_step": round(ms, 4),
           "tflops": round(algo / (ms * 1e-3) / 1e12, 2),
           "flops_per_step": algo, "forward_flops": fwd_flops,
           "backward_ms_per_step_kernels": round(bwd_ms, 4),
           "backward_tflops_kernels": round((bf["bwd_gemm"] + bf["bwd_attn_algorithmic"]) /
                                            (bwd_ms * 1e-3) / 1e12, 1),
           "per_kernel_tflops": rates, "per_kernel_roofline": kernel_fracs(rates),
           "finite": ok, "kernels": kern,
           "note": "step = kvp_train_forward + kvp_backward; TFLOP/s counts 3x the forward's "
                   "algorithmic FLOPs; attention kernels' figures count the products they execute "
                   "(S and dP recomputed), bwd_attn_algorithmic counts dV, dP, dQ, dK once"}
    log(f"[bench] train {ms:.3f} ms/step, {out['tflops']} TFLOP/s; backward kernels {bwd_ms:.3f} ms, "
        f"rates {rates}")
    return out


def bench_decode(w: ki.Workload, steps: int, warmup: int, alias_of=None):
    import torch
    from kvp_inputs import device as kd
    from paper_2608_15943_amd import binding as kb
    lens = w.lengths()
    B = w.batch
    max_len = int(lens.max())
    t0 = time.perf_counter()
    st = Stack(w, B, 1, w.kv_capacity, fill_npos=max_len, alias_of=alias_of)
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

def host_info():
    """Host cores, BLAS threads and CPU model, reported with every oracle figure."""
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count() or 1
    model = ""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return int(threads), {"os_cpu_count": os.cpu_count(), "blas_threads": int(threads), "cpu_model": model}


def oracle_weights(w: ki.Workload):
    from oracle import attention as oat
    ws = []
    for l in range(w.L):
        prod = w.tau[l] == l
        ws.append(oat.LayerWeights(ki.weight(w, ki.KIND_WQ, l),
                                   ki.weight(w, ki.KIND_WK, l) if prod else None,
                                   ki.weight(w, ki.KIND_WV, l) if prod else None,
                                   ki.weight(w, ki.KIND_WO, l)))
    return ws


def cpu_baseline(w: ki.Workload, s_sample: int):
    from oracle import attention as oat
    threads, host = host_info()
    ws = oracle_weights(w)
    x = ki.prefill_x(w, [0], np.arange(s_sample))[0]
    t0 = time.perf_counter()
    oat.stack_prefill(x, ws, w.tau, w.a, w.g, w.d_h, w.rope_base)
    dt = time.perf_counter() - t0
    flops = sum(prefill_flops(w, 1, s_sample).values())
    return {"value": round(flops / dt / 1e12, 6), "unit": "TFLOP/s", "cores": threads,
            "kind": "oracle",
            "sample": (f"sequence 0 of {w.batch}, " +
                       (f"all {s_sample} positions" if s_sample == w.seq else
                        f"first {s_sample} positions (causal prefix, exact)") +
                       f", all {w.L} layers, fp64 NumPy with host BLAS; {dt:.1f} s"),
            "host": host}


def cpu_baseline_decode(wd: ki.Workload, lens, sample: int = 0):
    """The oracle's decode step for one sequence of the batch through all layers (rows of a
    batch never interact, so one sequence is an exact sample); the time to regenerate its
    cache from the seeded generator is excluded and reported separately."""
    from oracle import attention as oat
    threads, host = host_info()
    L = int(lens[sample])
    t0 = time.perf_counter()
    caches = {p: (ki.cache_contents(wd, ki.KIND_KCACHE, p, sample, L),
                  ki.cache_contents(wd, ki.KIND_VCACHE, p, sample, L)) for p in wd.producers()}
    ws = oracle_weights(wd)
    x = ki.decode_x(wd, [sample])[0]
    t1 = time.perf_counter()
    oat.decode_step(x, L, ws, wd.tau, caches, wd.a, wd.g, wd.d_h, wd.rope_base)
    dt = time.perf_counter() - t1
    return {"value": round(1.0 / dt, 4), "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": (f"sequence {sample} of {wd.batch} ({L} cached positions), all {wd.L} layers, "
                       f"fp64 NumPy with host BLAS; {dt:.2f} s (cache regeneration "
                       f"{t1 - t0:.1f} s, not counted)"),
            "host": host}


def calibrate_copy():
    """A plain device-to-device copy of exactly 1 GiB, five times: rocprofv3's FETCH_SIZE and
    WRITE_SIZE for this kernel give the factor between the counters and true bytes."""
    import torch
    n = 1 << 30
    a = torch.empty(n, dtype=torch.uint8, device="cuda")
    a.fill_(1)
    b = torch.empty_like(a)
    for _ in range(5):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"calibration": "device copy", "bytes_read": n, "bytes_written": n, "launches": 5}))


ACHIEVABLE = {}


def achievable_peaks():
    """What this device delivers, measured with the library's calibration kernels
    (include/kvp_calib.h): a bf16 matrix-core loop with operands that change every
    instruction, and a streaming read of a 4 GiB buffer (16x the last-level cache).  Best of
    5 (matrix) / 10 (read) timed launches after 3 / 20 untimed ones, HIP events on the launch
    stream."""
    import torch
    from paper_2608_15943_amd import binding as kb
    st = torch.cuda.current_stream()
    sink = torch.zeros(64, dtype=torch.uint8, device="cuda")
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def best(launch, warm=3, reps=5):
        for _ in range(warm):   # the clocks ramp up under sustained load first
            launch()
        t = []
        for _ in range(reps):
            e0.record(st)
            launch()
            e1.record(st)
            e1.synchronize()
            t.append(e0.elapsed_time(e1))
        return min(t)
    iters = 20000
    flops = kb.kvp_calib_mfma_bf16(iters, sink.data_ptr(), st.cuda_stream)
    ms = best(lambda: kb.kvp_calib_mfma_bf16(iters, sink.data_ptr(), st.cuda_stream))
    n = 4 << 30
    buf = torch.empty(n // 8, dtype=torch.int64, device="cuda").random_()
    ms_r = best(lambda: kb.kvp_calib_stream_read(buf.data_ptr(), n, sink.data_ptr(), st.cuda_stream),
                warm=20, reps=10)
    del buf
    torch.cuda.empty_cache()
    ACHIEVABLE.update({
        "mfma_bf16_tflops": round(flops / (ms * 1e-3) / 1e12, 1),
        "hbm_read_gbs": round(n / (ms_r * 1e-3) / 1e9, 1),
        "method": "kvp_calib_mfma_bf16 (8 waves per CU, v_mfma_f32_32x32x16_bf16 on random bf16 "
                  "operands, 20000 x 16 per wave), best of 5 after 3; kvp_calib_stream_read (4 GiB), "
                  "best of 10 after 20"})
    return dict(ACHIEVABLE)


def mall_probe(sizes_mib=(32, 64, 128, 192, 256, 384, 512), trials: int = 5):
    """Does a second read of a buffer hit the 256 MB last-level (Infinity) cache?  For each
    size: read a 2 GiB buffer (evicts), time a read of the buffer (cold), time it again at
    once (re-read), read 64 MiB of other data, time it again; median of `trials`.  A consumer
    layer re-reading its producer's cache from that level is only worth a schedule change if
    the re-read is much faster than HBM."""
    import torch
    from paper_2608_15943_amd import binding as kb
    st = torch.cuda.current_stream()
    sink = torch.zeros(16, dtype=torch.uint8, device="cuda")
    flush = torch.empty(2 << 30, dtype=torch.uint8, device="cuda")
    other = torch.empty(64 << 20, dtype=torch.uint8, device="cuda")

    def rd(buf):
        _check = kb.lib().kvp_calib_stream_read(buf.data_ptr(), buf.numel(), sink.data_ptr(), st.cuda_stream)
        if _check != 0:
            raise RuntimeError(f"kvp_calib_stream_read failed ({_check})")

    def timed(buf):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(st)
        rd(buf)
        b.record(st)
        b.synchronize()
        return a.elapsed_time(b)

    out = {}
    for mib in sizes_mib:
        buf = torch.empty(mib << 20, dtype=torch.uint8, device="cuda")
        res = []
        for _ in range(trials):
            rd(flush)
            c, w = timed(buf), timed(buf)
            rd(other)
            res.append((c, w, timed(buf)))
        res.sort()
        c, w, wi = res[len(res) // 2]
        gb = (mib << 20) / 1e9
        out[f"{mib}MiB"] = {"cold_gbs": round(gb / (c * 1e-3)), "reread_gbs": round(gb / (w * 1e-3)),
                            "reread_after_64MiB_gbs": round(gb / (wi * 1e-3))}
        del buf
    return out


def kernel_fracs(tflops: dict, workload=None) -> dict:
    """Every MFMA kernel's algorithmic TFLOP/s against the datasheet and the measured peak, with
    the committed matrix-core counters of that kernel on that workload (mfma_counters_for)."""
    ach = ACHIEVABLE.get("mfma_bf16_tflops")
    return {k: {"tflops": v, "frac": round(v / PEAK_BF16_TFLOPS, 4),
                "frac_achievable": round(v / ach, 4) if ach else None,
                "mfma_counters": mfma_counters_for(k, workload) if workload else None}
            for k, v in tflops.items()}


def _committed(name, kernel, workload):
    """Entry kernel@workload of profiles/<name>, or None if there is none or the kernel's
    sources differ from the ones the counters were taken on."""
    import hashlib
    path = os.path.join(ROOT, "profiles", name)
    if not os.path.exists(path):
        return None
    with open(path) as f:
        ent = json.load(f).get(f"{kernel}@{workload}")
    if not ent:
        return None
    h = hashlib.sha1()
    for rel in ent["sources"]:
        src = os.path.join(ROOT, rel)
        if not os.path.exists(src):
            return None
        with open(src, "rb") as f:
            h.update(f.read())
    return ent if h.hexdigest() == ent["sources_sha1"] else None


def mfma_counters_for(kernel, workload):
    """The committed rocprofv3 matrix-core counters of this kernel on this workload
    (profiles/mfma.json, profiles/prefill_mfma_counters.md): the share of cycles its matrix cores
    were busy, the clock it ran at, and the datasheet fraction they imply (busy x clock / 2.4
    GHz), which corroborates the event-timed frac.  None if the sources changed since."""
    ent = _committed("mfma.json", kernel, workload)
    if not ent:
        return None
    return {"mfma_busy": ent["mfma_busy"], "clock_ghz": ent["clock_ghz"],
            "implied_frac": round(ent["mfma_busy"] * ent["clock_ghz"] / 2.4, 4),
            "bf16_flop_counted_per_dispatch": ent["bf16_flop_counted"]}


def roofline_entry(kernel, prof, per_unit, units_per_launch, peak, unit, bound, workload):
    """Algorithmic work per launch (per-unit figure x units one launch processes) over the
    kernel's average launch time, measured with HIP events on the launch stream."""
    n, t = prof[kernel]
    per_launch = per_unit * units_per_launch
    achieved = per_launch / (t / n * 1e-3) / (1e12 if unit == "TFLOP/s" else 1e9)
    ent = {"bound": bound, "kernel": kernel, "achieved": round(achieved, 2), "peak": peak,
           "unit": unit, "frac": round(achieved / peak, 4), "traffic": traffic_for(kernel, workload),
           **({"mfma_counters": mfma_counters_for(kernel, workload)} if bound == "mfma" else {}),
           "work_per_launch": per_launch, "avg_launch_ms": round(t / n, 5)}
    # The same figure against what this device measurably delivers (achievable_peaks).
    ach = ACHIEVABLE.get("mfma_bf16_tflops" if unit == "TFLOP/s" else "hbm_read_gbs")
    if ach:
        ent["peak_achievable"] = ach
        ent["frac_achievable"] = round(achieved / ach, 4)
    return ent


def traffic_for(kernel, workload):
    """HBM bytes per launch from the committed FETCH_SIZE / WRITE_SIZE counter runs (scaled by
    the factor a plain copy of known size gives) of this kernel on this workload, or None if
    there is none or the kernel's sources differ from the ones the counters were taken on."""
    ent = _committed("traffic.json", kernel, workload)
    return ent["bytes_per_launch"] if ent else None


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-decode", action="store_true")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--no-unshared", action="store_true")
    ap.add_argument("--cpu-seq", type=int, default=4096)
    ap.add_argument("--no-extra", action="store_true",
                    help="skip the 70B-shaped prefill and the ragged 128K decode lines")
    ap.add_argument("--no-calib", action="store_true",
                    help="skip the achievable-peak calibration (no frac_achievable figures)")
    ap.add_argument("--no-train", action="store_true", help="skip the training-step line")
    ap.add_argument("--only", choices=["prefill", "prefill_70b", "decode", "decode_128k", "calib", "tiny",
                                       "train", "decode_capacity", "mall", "decode_graph", "prefill_paged"],
                    help="run one workload only and print its entry (for profiling)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a plain 1 GiB device copy (rocprofv3 counter calibration)")
    args = ap.parse_args()
    if args.calibrate_copy:
        calibrate_copy()
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (the KV-shared block is measured on one GPU's share; "
              f"more GPUs would each run their own stage or batch share); --gpus {args.gpus} is not supported",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2608_15943_amd import binding as kb
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    kb.lib()   # fail loudly if the HIP library is missing
    if args.only == "calib":
        print(json.dumps({"only": "calib", **achievable_peaks()}), flush=True)
        return
    if args.only == "mall":
        print(json.dumps({"only": "mall", **mall_probe()}), flush=True)
        return
    if not args.no_calib and not args.only:
        log(f"[bench] achievable peaks {achievable_peaks()}")
    if args.only:
        steps_d, warm_d = max(3, args.steps // 2), max(1, args.warmup // 2)
        if args.only == "prefill_70b":
            out = bench_70b(args.steps, args.warmup)
        elif args.only == "decode":
            out = decode_entry(ki.decode_32k(), steps_d, warm_d)
        elif args.only == "decode_128k":
            out = decode_entry(ki.decode_128k_ragged(), steps_d, warm_d)
        elif args.only == "train":
            out = train_entry(ki.stage_share_prefill(), steps_d, warm_d)
        elif args.only == "decode_capacity":
            out = capacity_entry(steps_d, warm_d)
        elif args.only == "tiny":
            out = tiny_entry(args.steps, args.warmup)
        elif args.only == "decode_graph":
            out = graph_entry(args.steps, args.warmup)
        elif args.only == "prefill_paged":
            out = paged_prefill_entry(args.steps, args.warmup)
        else:
            w = ki.stage_share_prefill()
            ms, prof, finite = bench_prefill(w, args.steps, args.warmup)
            out = {"workload": w.name, "ms_per_step": round(ms, 4), "finite": finite,
                   "kernels": {k: {"launches": n, "avg_ms": round(t / n, 5)} for k, (n, t) in prof.items()}}
        print(json.dumps({"only": args.only, **out}), flush=True)
        return

    w = ki.stage_share_prefill()
    log(f"[bench] prefill {w.name} steps={args.steps} warmup={args.warmup}")
    ms, prof, finite = bench_prefill(w, args.steps, args.warmup)
    flops = prefill_flops(w, w.batch, w.seq)
    total = sum(flops.values())
    value = total / (ms * 1e-3) / 1e12
    kernels = {k: {"launches": n, "avg_ms": round(t / n, 5)} for k, (n, t) in prof.items()}
    dom = max(("qkv_gemm", "flash_attn", "oproj_gemm"), key=lambda k: prof.get(k, (0, 0.0))[1])
    n_l = prof[dom][0]
    roofline = roofline_entry(dom, prof, flops[dom] / w.L, w.L * args.steps / n_l,
                              PEAK_BF16_TFLOPS, "TFLOP/s", "mfma", w.name)
    roofline["per_unit"] = "algorithmic FLOPs of one layer of the stack (batch 4 x 4096 tokens)"
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
        "achievable": dict(ACHIEVABLE) or None,
        "kernels": kernels,
        "per_kernel_tflops": {k: round(flops[k] * args.steps / prof[k][1] / 1e9, 1)
                              for k in flops if k in prof},
        "finite": finite,
    }
    result["per_kernel_roofline"] = kernel_fracs(result["per_kernel_tflops"], w.name)

    if not args.no_unshared:
        ident = list(range(w.L))
        ms_u, _, _ = bench_prefill(w, args.steps, args.warmup, tau=ident)
        ideal = sum(prefill_flops(w, w.batch, w.seq, ident).values()) / total
        result["shared_vs_unshared"] = {"prefill_speedup": round(ms_u / ms, 4),
                                        "prefill_ideal": round(ideal, 4),
                                        "unshared_ms_per_step": round(ms_u, 4)}
        log(f"[bench] identity map {ms_u:.3f} ms/step (speedup {ms_u / ms:.4f}, ideal {ideal:.4f})")

    if not args.no_extra:
        result["prefill_70b_stage"] = bench_70b(args.steps, args.warmup, unshared=not args.no_unshared,
                                                cpu=not args.no_cpu)
        result["tiny_fp32"] = tiny_entry(args.steps, args.warmup)
        result["prefill_paged"] = paged_prefill_entry(args.steps, args.warmup)

    if not args.no_train:
        result["train"] = train_entry(w, max(3, args.steps // 2), max(1, args.warmup // 2))

    if not args.no_decode:
        steps_d, warm_d = max(3, args.steps // 2), max(1, args.warmup // 2)
        wd = ki.decode_32k()
        result["decode"] = decode_entry(wd, steps_d, warm_d)
        if not args.no_cpu:
            log("[bench] oracle CPU baseline (decode, one sequence)")
            result["decode"]["cpu_baseline"] = cpu_baseline_decode(wd, wd.lengths())
        if not args.no_unshared:
            # Identity map: every layer owns a cache.  All 32 caches (275 GB) do not fit
            # beside the rest, so former consumers reuse their former producer's memory;
            # every layer still reads and appends its own full cache.
            wi = wd.with_map(list(range(wd.L)), "-identity")
            u = decode_entry(wi, steps_d, warm_d, alias_of={l: wd.tau[l] for l in range(wd.L)
                                                            if wd.tau[l] != l})
            sh, un = result["decode"]["step_ms_spread"], u["step_ms_spread"]
            result["decode"]["shared_vs_unshared"] = {
                "step_speedup": round(u["ms_per_step"] / result["decode"]["ms_per_step"], 4),
                "step_speedup_range": [round(un["min"] / sh["max"], 4), round(un["max"] / sh["min"], 4)],
                "ideal": round(sum(decode_bytes(wi, wi.lengths()).values()) /
                               sum(decode_bytes(wd, wd.lengths()).values()), 4),
                "unshared_ms_per_step": u["ms_per_step"], "unshared_step_ms_spread": un,
                "aliased": True,
                "alias_map": {str(l): wd.tau[l] for l in range(wd.L) if wd.tau[l] != l},
                "alias_note": "the 32 unshared caches (275 GB) do not fit beside the rest, so each "
                              "former consumer's slot is the memory of its former producer's; every "
                              "layer still appends and reads a full cache of its own length",
                "kv_cache_bytes_shared": kv_bytes(wd), "kv_cache_bytes_unshared": kv_bytes(wi)}
        if not args.no_extra:
            w4 = ki.decode_128k_ragged()
            result["decode_ragged_128k"] = decode_entry(w4, steps_d, warm_d)
            if not args.no_unshared:
                # Identity map: all 32 layers own a cache (137 GB at 128K capacity, fits).
                w4i = w4.with_map(list(range(w4.L)), "-identity")
                u4 = decode_entry(w4i, steps_d, warm_d)
                sh, un = result["decode_ragged_128k"]["step_ms_spread"], u4["step_ms_spread"]
                result["decode_ragged_128k"]["shared_vs_unshared"] = {
                    "step_speedup": round(u4["ms_per_step"] / result["decode_ragged_128k"]["ms_per_step"], 4),
                    "step_speedup_range": [round(un["min"] / sh["max"], 4), round(un["max"] / sh["min"], 4)],
                    "ideal": round(sum(decode_bytes(w4i, w4i.lengths()).values()) /
                                   sum(decode_bytes(w4, w4.lengths()).values()), 4),
                    "unshared_ms_per_step": u4["ms_per_step"], "unshared_step_ms_spread": un,
                    "aliased": False,
                    "kv_cache_bytes_shared": kv_bytes(w4), "kv_cache_bytes_unshared": kv_bytes(w4i)}
            if not args.no_cpu:
                log("[bench] oracle CPU baseline (ragged 128K decode, the shortest sequence)")
                l4 = w4.lengths()
                result["decode_ragged_128k"]["cpu_baseline"] = cpu_baseline_decode(w4, l4, int(np.argmin(l4)))
            result["decode_capacity"] = capacity_entry(steps_d, warm_d)
            result["decode_graph"] = graph_entry(args.steps, args.warmup)

    if not args.no_cpu:
        log(f"[bench] oracle CPU baseline ({args.cpu_seq} positions of one sequence)")
        result["cpu_baseline"] = cpu_baseline(w, args.cpu_seq)

    result["workloads"] = workload_table(result)
    print(json.dumps(result), flush=True)


def workload_table(r):
    """One row per workload of the run: step time, rate, roofline fraction of the dominant
    kernel, shared-vs-unshared ratio and the oracle's rate, gathered from the entries above."""
    def cpu(e):
        c = e.get("cpu_baseline")
        return None if not c else {"value": c["value"], "unit": c["unit"], "cores": c["cores"],
                                   **({"extrapolated": True} if c.get("extrapolated") else {})}
    rows = {r["config"]["workload"]: {
        "ms_per_step": r["ms_per_step"], "rate": r["value"], "unit": r["unit"],
        "roofline_frac": r["roofline"]["frac"], "roofline_kernel": r["roofline"]["kernel"],
        "shared_vs_unshared": (r.get("shared_vs_unshared") or {}).get("prefill_speedup"), "cpu_baseline": cpu(r)}}
    if "tiny_fp32" in r:
        e = r["tiny_fp32"]
        rows[e["workload"]] = {"ms_per_step": e["ms_per_step"], "rate": e["tflops"], "unit": "TFLOP/s",
                               "roofline_frac": None, "roofline_kernel": "launch-bound: time only",
                               "shared_vs_unshared": None, "cpu_baseline": cpu(e)}
    if "prefill_70b_stage" in r:
        e = r["prefill_70b_stage"]
        rows[e["workload"]] = {"ms_per_step": e["ms_per_step"], "rate": e["tflops"], "unit": "TFLOP/s",
                               "roofline_frac": e["roofline"]["frac"], "roofline_kernel": e["roofline"]["kernel"],
                               "shared_vs_unshared": (e.get("shared_vs_unshared") or {}).get("prefill_speedup"),
                               "cpu_baseline": cpu(e)}
    for k in ("decode", "decode_ragged_128k"):
        if k in r:
            e = r[k]
            rows[e["workload"]] = {"ms_per_step": e["ms_per_step"], "rate": e["tokens_per_s"], "unit": "tokens/s",
                                   "hbm_gbs": e["hbm_gbs"], "hbm_frac": e["hbm_frac"],
                                   "roofline_frac": e["roofline"]["frac"], "roofline_kernel": e["roofline"]["kernel"],
                                   "shared_vs_unshared": (e.get("shared_vs_unshared") or {}).get("step_speedup"),
                                   "cpu_baseline": cpu(e)}
    return rows


def kv_bytes(w: ki.Workload) -> int:
    """Resident KV-cache bytes of a decode workload (K and V^T slots of every producer)."""
    return len(w.producers()) * 2 * w.batch * w.g * w.kv_capacity * w.d_h * 2


def decode_entry(wd: ki.Workload, steps: int, warmup: int, alias_of=None):
    log(f"[bench] decode {wd.name}")
    dms, dprof, dfin, lens = bench_decode(wd, steps, warmup, alias_of=alias_of)
    spread = step_spread()
    db = decode_bytes(wd, lens)
    dtotal = sum(db.values())
    n_a = dprof["dec_attn"][0]
    ctx = int(np.sum(lens.astype(np.int64) + 1))
    rl = roofline_entry("dec_attn", dprof, 2 * wd.g * wd.d_h * 2, ctx * wd.L * steps / n_a,
                        PEAK_HBM_GBS, "GB/s", "hbm", wd.name)
    rl["per_unit"] = "bytes of K and V read for one cached position of one layer (g*d_h*2*2)"
    out = {
        "workload": wd.name, "batch": wd.batch, "context": [int(lens.min()), int(lens.max())],
        "map": wd.tau, "tokens_per_s": round(wd.batch / (dms * 1e-3), 2),
        "ms_per_step": round(dms, 4), "step_ms_spread": spread,
        "hbm_gbs": round(dtotal / (dms * 1e-3) / 1e9, 1),
        "hbm_frac": round(dtotal / (dms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
        "hbm_frac_achievable": (round(dtotal / (dms * 1e-3) / 1e9 / ACHIEVABLE["hbm_read_gbs"], 4)
                                if ACHIEVABLE.get("hbm_read_gbs") else None),
        "bytes_per_step": dtotal, "kv_cache_bytes": kv_bytes(wd), "finite": dfin,
        "roofline": rl,
        "kernels": {k: {"launches": n, "avg_ms": round(t / n, 5)} for k, (n, t) in dprof.items()},
    }
    log(f"[bench] decode {dms:.3f} ms/step, {out['tokens_per_s']} tok/s, "
        f"attention {rl['achieved']:.0f} GB/s")
    return out


PAGE = 64


def paged_decode(w: ki.Workload, lens, table, n_pages: int, steps: int, warmup: int):
    """One decode step over len(lens) sequences whose caches live in n_pages-page pools under
    `table` (host int32 [B][row]), timed like bench_decode."""
    import torch
    from kvp_inputs import device as kd
    from paper_2608_15943_amd import binding as kb
    B, row = len(lens), table.shape[1]
    t0 = time.perf_counter()
    st = Stack(w, B, 1, PAGE, slots=False)
    pools = []
    tab_t = torch.from_numpy(np.ascontiguousarray(table)).cuda()
    lens_t = torch.tensor(lens, dtype=torch.int32, device="cuda")
    for l in w.producers():
        K = torch.empty((w.g, n_pages, PAGE, w.d_h), dtype=torch.bfloat16, device="cuda")
        V = torch.empty((w.g, n_pages, w.d_h, PAGE), dtype=torch.bfloat16, device="cuda")
        kd.fill_cache_pages(w, l, K.data_ptr(), V.data_ptr(), tab_t.data_ptr(), row, n_pages, lens_t.data_ptr(), B)
        st.model.kvp_set_kv_pool(l, K.data_ptr(), V.data_ptr(), n_pages)
        pools.append((K, V))
    torch.cuda.synchronize()
    log(f"[bench] paged decode {w.name} B={B} setup {time.perf_counter() - t0:.1f}s "
        f"({torch.cuda.memory_allocated() / 2**30:.1f} GiB resident)")
    x = torch.empty((B, w.h), dtype=torch.bfloat16, device="cuda")
    kd.fill_decode_x(w, x.data_ptr(), B)
    y = torch.empty_like(x)
    max_len = int(np.max(lens))
    n = st.model.kvp_workspace_size(kb.KVP_PHASE_DECODE, B)
    ws = torch.empty(n, dtype=torch.uint8, device="cuda")
    cs = torch.cuda.current_stream().cuda_stream

    def run():
        st.model.kvp_decode_step_paged(x.data_ptr(), lens_t.data_ptr(), max_len, tab_t.data_ptr(), row,
                                       y.data_ptr(), B, ws.data_ptr(), n, cs)

    ms, prof = time_steps(run, st.model, steps, warmup)
    fin = bool(torch.isfinite(y.float()).all().item())
    del st, pools, x, y, ws, tab_t, lens_t
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return ms, prof, fin


def capacity_scenario(base: ki.Workload, budget: int, max_rows: int, steps: int, warmup: int):
    """Admit the sequences of base's ragged length stream in order until a budget-sized pool
    is full (each needs len + 1 positions), for the shared map and the identity map; then
    time one decode step over all admitted sequences on pages."""
    import dataclasses

    from paper_2608_15943_amd import binding as kb
    stream = dataclasses.replace(base, batch=max_rows).lengths()
    row = base.kv_capacity // PAGE
    out = {"context_distribution": [base.ctx_lo, base.ctx_hi], "maps": {}}
    for label, w in (("shared", base), ("identity", base.with_map(list(range(base.L)), "-identity"))):
        nprod = len(w.producers())
        page_bytes = 2 * PAGE * w.g * w.d_h * 2
        n_pages = budget // (page_bytes * nprod)
        slot_seqs = budget // (nprod * 2 * w.g * w.kv_capacity * w.d_h * 2)
        pager = kb.Pager(n_pages, max_rows, row)
        B = 0
        while B < max_rows and pager.try_reserve(B, int(stream[B]) + 1):
            B += 1
        lens = stream[:B]
        tab = pager.rows(list(range(B)))
        used = n_pages - pager.free_pages()
        pager.close()
        log(f"[bench] capacity {w.name} {label}: {B} sequences on {used}/{n_pages} pages per producer "
            f"(contiguous slots: {slot_seqs})")
        wb = dataclasses.replace(w, batch=B)
        ms, prof, fin = paged_decode(wb, lens, tab, n_pages, steps, warmup)
        db = decode_bytes(w, lens)
        ctx = int(np.sum(lens.astype(np.int64) + 1))
        n_a = prof["dec_attn"][0]
        rl = roofline_entry("dec_attn", prof, 2 * w.g * w.d_h * 2, ctx * w.L * steps / n_a,
                            PEAK_HBM_GBS, "GB/s", "hbm", w.name + "-paged")
        rl["per_unit"] = "bytes of K and V read for one cached position of one layer (g*d_h*2*2)"
        out["maps"][label] = {
            "producers": nprod, "pages_per_producer": int(n_pages), "pages_used": int(used),
            "max_sequences_paged": B, "max_sequences_contiguous": int(slot_seqs),
            "resident_tokens": ctx, "context": [int(lens.min()), int(lens.max())],
            "ms_per_step": round(ms, 4), "tokens_per_s": round(B / (ms * 1e-3), 2),
            "hbm_gbs": round(sum(db.values()) / (ms * 1e-3) / 1e9, 1), "finite": fin, "roofline": rl,
            "kernels": {k: {"launches": c, "avg_ms": round(t / c, 5)} for k, (c, t) in prof.items()}}
        log(f"[bench] capacity {label}: {ms:.2f} ms/step, {B / (ms * 1e-3):.1f} tok/s, "
            f"attention {rl['achieved']:.0f} GB/s")
    sh, idn = out["maps"]["shared"], out["maps"]["identity"]
    out["shared_vs_identity"] = {
        "sequences_paged": round(sh["max_sequences_paged"] / max(idn["max_sequences_paged"], 1), 3),
        "sequences_contiguous": round(sh["max_sequences_contiguous"] / max(idn["max_sequences_contiguous"], 1), 3),
        "tokens_per_s": round(sh["tokens_per_s"] / idn["tokens_per_s"], 4)}
    return out


def capacity_entry(steps: int, warmup: int, budget_gib: float = 160.0):
    """Capacity-driven decode (paged KV storage): with budget_gib of HBM for the KV cache, how
    many sequences fit, shared vs identity map, in 64-position pages and in contiguous slots
    at the stream's capacity, and one decode step over all of them.  Two length streams of
    the 32-layer model: ragged 64K-128K (capacity 128K) and ragged 8K-16K (capacity 16K;
    more than 64 sequences, so decode runs in 64-sequence chunks).  Also the cost of paging
    itself: the 8-sequence ragged workload on pages against the same workload on slots."""
    import dataclasses

    from paper_2608_15943_amd import binding as kb
    base = ki.decode_128k_ragged()
    budget = int(budget_gib * 2**30)
    out = {"workload": base.name + "-capacity", "kv_budget_bytes": budget, "page_positions": PAGE}
    out.update(capacity_scenario(base, budget, 64, steps, warmup))
    short = dataclasses.replace(base, name="decode-32L-d4096-gqa32x8-ctx8k-16k", ctx_lo=8192, ctx_hi=16383,
                                kv_capacity=16384)
    out["ctx_8k_16k"] = capacity_scenario(short, budget, 1024, steps, warmup)
    # Paging overhead: the 8-sequence ragged workload, pages vs slots.
    lens8 = base.lengths()
    row = base.kv_capacity // PAGE
    pager = kb.Pager(int(np.sum((lens8.astype(np.int64) + PAGE) // PAGE)), base.batch, row)
    for b, L in enumerate(lens8):
        pager.reserve(b, int(L) + 1)
    tab8 = pager.rows(list(range(base.batch)))
    pager.close()
    ms_p, _, _ = paged_decode(base, lens8, tab8, int(tab8.max()) + 1, steps, warmup)
    ms_s, _, _, _ = bench_decode(base, steps, warmup)
    out["paged_vs_slots_b8"] = {"paged_ms_per_step": round(ms_p, 4), "slots_ms_per_step": round(ms_s, 4),
                                "ratio": round(ms_p / ms_s, 4)}
    log(f"[bench] 8-sequence ragged decode: pages {ms_p:.3f} ms, slots {ms_s:.3f} ms")
    return out


def paged_prefill_entry(steps: int, warmup: int):
    """Cost of paging in prefill: the 8-layer stage share (B 4 x S 4096) on contiguous slots
    and on pages (a seeded permutation of a pool of exactly the pages needed), same model."""
    import torch
    from kvp_inputs import device as kd
    from paper_2608_15943_amd import binding as kb
    w = ki.stage_share_prefill()
    B, S = w.batch, w.seq
    st = Stack(w, B, S, w.kv_capacity)
    row = S // PAGE
    n_pages = B * row
    tab = torch.from_numpy(np.random.RandomState(1).permutation(n_pages).astype(np.int32).reshape(B, row)).cuda()
    pools = []
    for l in w.producers():
        K = torch.empty((w.g, n_pages, PAGE, w.d_h), dtype=torch.bfloat16, device="cuda")
        V = torch.empty((w.g, n_pages, w.d_h, PAGE), dtype=torch.bfloat16, device="cuda")
        st.model.kvp_set_kv_pool(l, K.data_ptr(), V.data_ptr(), n_pages)
        pools.append((K, V))
    x = torch.empty((B, S, w.h), dtype=torch.bfloat16, device="cuda")
    kd.fill_prefill_x(w, x.data_ptr(), B, S)
    y = torch.empty_like(x)
    yp = torch.empty_like(x)
    n = st.model.kvp_workspace_size(kb.KVP_PHASE_PREFILL, B, S)
    ws = torch.empty(n, dtype=torch.uint8, device="cuda")
    cs = torch.cuda.current_stream().cuda_stream
    ms_s, prof_s = time_steps(lambda: st.model.kvp_prefill(x.data_ptr(), y.data_ptr(), B, S, ws.data_ptr(), n, cs),
                              st.model, steps, warmup)
    ms_p, prof_p = time_steps(lambda: st.model.kvp_prefill_paged(x.data_ptr(), yp.data_ptr(), B, S, tab.data_ptr(),
                                                                 row, ws.data_ptr(), n, cs),
                              st.model, steps, warmup)
    same = bool(torch.equal(y, yp))
    avg = lambda prof, k: round(prof[k][1] / prof[k][0], 5)
    out = {"workload": w.name, "slots_ms_per_step": round(ms_s, 4), "pages_ms_per_step": round(ms_p, 4),
           "ratio": round(ms_p / ms_s, 4), "output_equal": same,
           "kernels_avg_ms": {k: {"slots": avg(prof_s, k), "pages": avg(prof_p, k)}
                              for k in ("qkv_gemm", "flash_attn", "oproj_gemm")}}
    log(f"[bench] paged prefill {ms_p:.3f} ms vs slots {ms_s:.3f} ms (equal outputs: {same})")
    del st, pools, x, y, yp, ws, tab
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return out


def graph_entry(steps: int, warmup: int, B: int = 8, ctx: int = 4096):
    """Launch-bound decode: the 32-layer model (shared map of the 32K workload) at a small
    batch and short context, 160 launches per step, eager against the same step captured
    once into a HIP graph and replayed."""
    import dataclasses

    import torch
    from kvp_inputs import device as kd
    from paper_2608_15943_amd import binding as kb
    w = dataclasses.replace(ki.decode_32k(), name=f"decode-32L-d4096-gqa32x8-b{B}-ctx{ctx}", batch=B, ctx=ctx,
                            kv_capacity=ctx + PAGE)
    st = Stack(w, B, 1, w.kv_capacity, fill_npos=ctx)
    x = torch.empty((B, w.h), dtype=torch.bfloat16, device="cuda")
    kd.fill_decode_x(w, x.data_ptr(), B)
    y = torch.empty_like(x)
    lens_t = torch.full((B,), ctx, dtype=torch.int32, device="cuda")
    n = st.model.kvp_workspace_size(kb.KVP_PHASE_DECODE, B)
    ws = torch.empty(n, dtype=torch.uint8, device="cuda")

    def run():
        st.model.kvp_decode_step(x.data_ptr(), lens_t.data_ptr(), ctx, y.data_ptr(), B, ws.data_ptr(), n,
                                 torch.cuda.current_stream().cuda_stream)

    def timed(f):
        for _ in range(warmup):
            f()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            f()
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) * 1e3 / steps

    ms_eager = timed(run)
    ref = y.clone()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        run()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        run()
    torch.cuda.synchronize()
    ms_graph = timed(g.replay)
    same = bool(torch.equal(y, ref))
    out = {"workload": w.name, "batch": B, "context": ctx, "launches_per_step": 5 * w.L,
           "eager_ms_per_step": round(ms_eager, 4), "graph_ms_per_step": round(ms_graph, 4),
           "speedup": round(ms_eager / ms_graph, 4), "tokens_per_s_graph": round(B / (ms_graph * 1e-3), 1),
           "graph_output_equals_eager": same}
    log(f"[bench] decode graph {w.name}: eager {ms_eager:.3f} ms, graph {ms_graph:.3f} ms")
    del g, st, x, y, ws, lens_t
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return out


def bench_70b(steps: int, warmup: int, unshared: bool = False, cpu: bool = False):
    """The 70B-shaped stage: its map comes from the C++ planner (Algorithm 1) on the
    stage-tail-heavy synthetic FLOPs of 80 layers over 8 stages, each stage's first layer
    kept; the stage run on this GPU is the last one.  unshared: also time the identity map
    (every layer a producer); cpu: the oracle on a layer subset (see cpu_baseline_70b)."""
    from paper_2608_15943_amd import binding as kb
    Lw = 80
    t0 = time.perf_counter()
    f0, f1 = kb.kvp_layer_flops(1, 8192, 8192, 64, 8, causal=True)
    plan = kb.kvp_plan_fir([l // 10 for l in range(Lw)], [f0] * Lw, [f1] * Lw, 0.3 * 10 * f0, 0.05,
                           admissible=[l % 10 != 0 for l in range(Lw)])
    tau = kb.kvp_map_from_mask(plan["z"])
    plan_us = (time.perf_counter() - t0) * 1e6
    local = [t - 70 for t in tau[70:]]
    w5 = ki.stage_70b_prefill(local)
    log(f"[bench] prefill {w5.name} map {local} (planner {plan_us:.0f} us, FIR {plan['fir']:.4f})")
    steps5 = max(3, steps // 2)
    ms5, prof5, fin5 = bench_prefill(w5, steps5, max(1, warmup // 2))
    spread5 = step_spread()
    fl5 = prefill_flops(w5, w5.batch, w5.seq)
    dom5 = max(("qkv_gemm", "flash_attn", "oproj_gemm"), key=lambda k: prof5.get(k, (0, 0.0))[1])
    rl = roofline_entry(dom5, prof5, fl5[dom5] / w5.L, w5.L * steps5 / prof5[dom5][0],
                        PEAK_BF16_TFLOPS, "TFLOP/s", "mfma", w5.name)
    rl["per_unit"] = "algorithmic FLOPs of one layer (1 x 8192 tokens)"
    out = {"workload": w5.name, "map": local, "planner": {"fir": plan["fir"],
                                                          "n_converted": plan["n_converted"],
                                                          "host_us": round(plan_us, 1)},
           "tflops": round(sum(fl5.values()) / (ms5 * 1e-3) / 1e12, 2),
           "ms_per_step": round(ms5, 4), "step_ms_spread": spread5, "finite": fin5, "roofline": rl,
           "kernels": {k: {"launches": n, "avg_ms": round(t / n, 5)} for k, (n, t) in prof5.items()},
           "per_kernel_tflops": {k: round(fl5[k] * steps5 / prof5[k][1] / 1e9, 1)
                                 for k in fl5 if k in prof5}}
    out["per_kernel_roofline"] = kernel_fracs(out["per_kernel_tflops"], w5.name)
    log(f"[bench] 70B stage {ms5:.3f} ms/step, {out['tflops']} TFLOP/s")
    if unshared:
        ident = list(range(w5.L))
        ms_u, _, _ = bench_prefill(w5, steps5, max(1, warmup // 2), tau=ident)
        sp_u = step_spread()
        ideal = sum(prefill_flops(w5, w5.batch, w5.seq, ident).values()) / sum(fl5.values())
        out["shared_vs_unshared"] = {"prefill_speedup": round(ms_u / ms5, 4), "prefill_ideal": round(ideal, 4),
                                     "speedup_range": [round(sp_u["min"] / spread5["max"], 4),
                                                       round(sp_u["max"] / spread5["min"], 4)],
                                     "unshared_ms_per_step": round(ms_u, 4)}
        log(f"[bench] 70B stage identity map {ms_u:.3f} ms/step (speedup {ms_u / ms5:.4f}, ideal {ideal:.4f})")
    if cpu:
        log("[bench] oracle CPU baseline (70B-shaped stage, layer subset)")
        out["cpu_baseline"] = cpu_baseline_70b(w5)
    return out


def cpu_baseline_70b(w5: ki.Workload, s_sample: int = 2048):
    """The oracle on a bounded sample of the 70B-shaped stage: its producer (layer 0) and one
    consumer (the last layer, fed the producer's output and reading its K, V) over the first
    s_sample positions of the sequence (a causal prefix is an exact sample of those rows).
    The rate is the sample's algorithmic FLOPs over the oracle's time; applied to the whole
    stage it extrapolates (the oracle's attention cost grows with the sequence length)."""
    from oracle import attention as oat
    threads, host = host_info()
    sub = ki.Workload(**{**w5.__dict__, "L": 2, "tau": [0, 0]})
    wts = [oat.LayerWeights(ki.weight(w5, ki.KIND_WQ, 0), ki.weight(w5, ki.KIND_WK, 0),
                            ki.weight(w5, ki.KIND_WV, 0), ki.weight(w5, ki.KIND_WO, 0)),
           oat.LayerWeights(ki.weight(w5, ki.KIND_WQ, w5.L - 1), None, None,
                            ki.weight(w5, ki.KIND_WO, w5.L - 1))]
    x = ki.prefill_x(w5, [0], np.arange(s_sample))[0]
    t0 = time.perf_counter()
    oat.stack_prefill(x, wts, [0, 0], w5.a, w5.g, w5.d_h, w5.rope_base)
    dt = time.perf_counter() - t0
    flops = sum(prefill_flops(sub, 1, s_sample).values())
    rate = flops / dt
    return {"value": round(rate / 1e12, 6), "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
            "sample": (f"layers 0 (producer) and {w5.L - 1} (consumer of layer 0) on positions "
                       f"[0, {s_sample}) of the sequence, fp64 NumPy with host BLAS; {dt:.1f} s"),
            "extrapolated": True,
            "extrapolated_ms_per_step": round(sum(prefill_flops(w5, w5.batch, w5.seq).values()) / rate * 1e3, 1),
            "host": host}


def tiny_entry(steps: int, warmup: int):
    """The tiny fp32 stack (4 layers, d_model 256, 4 x 64 heads, S 128, map [0, 0, 2, 2]): every
    step on the vector ALUs in fp32; launch-bound, so only its time is reported (no roofline),
    next to the oracle's time for the same stack on the host."""
    from oracle import attention as oat
    w = ki.tiny_fp32()
    ms, prof, fin = bench_prefill(w, steps, warmup)
    fl = sum(prefill_flops(w, w.batch, w.seq).values())
    threads, host = host_info()
    wts = oracle_weights(w)
    x = ki.prefill_x(w, [0], np.arange(w.seq))[0]
    reps = 20
    t0 = time.perf_counter()
    for _ in range(reps):
        oat.stack_prefill(x, wts, w.tau, w.a, w.g, w.d_h, w.rope_base)
    dt = (time.perf_counter() - t0) / reps
    return {"workload": w.name, "dtype": "f32", "ms_per_step": round(ms, 4), "step_ms_spread": step_spread(),
            "tflops": round(fl / (ms * 1e-3) / 1e12, 4), "flops_per_step": fl, "finite": fin,
            "bound": "launch", "launches_per_step": sum(n for n, _ in prof.values()) // max(1, steps),
            "kernels": {k: {"launches": n, "avg_ms": round(t / n, 5)} for k, (n, t) in prof.items()},
            "cpu_baseline": {"value": round(fl / dt / 1e12, 6), "unit": "TFLOP/s", "cores": threads,
                             "kind": "oracle", "ms_per_step": round(dt * 1e3, 3),
                             "sample": f"the whole stack (sequence of {w.seq}), fp64 NumPy, mean of {reps} runs",
                             "host": host}}


if __name__ == "__main__":
    main()
