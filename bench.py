#!/usr/bin/env python3
"""Benchmark of the H2O chunk step on one MI355X.

Default workload: token generation, B=8, Hq=32, Hkv=8, d=64, M=4096, T=1,
bf16. One bench step is one token step (h2o_chunk_step: attention, score
accumulation, eviction and insert) for each of 8 independent layer states, so the 8 x 69 MB
working set exceeds the 256 MB Infinity Cache and the step streams from HBM.
Consecutive token steps (each with its own query, new key and value, drawn
for the workload's 16-step trajectory) are captured in one HIP graph, up to 16
steps of 8 layer states, and the graph is replayed so that exactly --steps
token steps are timed; ``value`` is algorithmic bytes per second (GB/s) over
the timed steps.

The chunked-prefill shapes (d=128: B1 Hq32 Hkv8 M8192 T1024; B4 Hq32 Hkv8
M32768 T512; B2 Hq28 Hkv4 M16384 T2048) are timed too and reported under
"prefill" as TFLOP/s of algorithmic attention work W = 4 d P B Hq,
P = T*M + T(T+1)/2. "insert_first" times the paper's own order of a step
(insert the chunk, then attend with the token-position mask) on the same
shapes, with P = (M - T)*T + T(T+1)/2 there.

Prints one JSON line. ``--gpus N`` with N > 1 exits: the benchmark runs on one GPU.
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

METRIC = "H2O SDPA TFLOP/s (% bf16 MFMA peak) prefill; decode HBM GB/s (% peak)"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
LAYERS = 8
PREFILL = ["prefill_bf16", "longcache_bf16", "gqa7_bf16"]


def decode_step_bytes(w) -> int:
    """Algorithmic HBM bytes of one token step of one layer state."""
    kv = 2 * w.B * w.Hkv * w.M * w.d * 2           # K and V cache read once
    q_out = 2 * w.B * w.Hq * w.T * w.d * 2         # q read, out written
    new = 4 * w.B * w.Hkv * w.T * w.d * 2          # k_new/v_new read and written to the cache
    scores = 2 * w.B * w.Hkv * w.M * 4             # scores read and written once
    return kv + q_out + new + scores


def decode_split_bytes(w) -> int:
    """Algorithmic bytes of one launch of the decode split kernel: the cache
    rows it streams plus the queries."""
    return 2 * w.B * w.Hkv * w.M * w.d * 2 + w.B * w.Hq * w.d * 2


def attention_flops(w) -> float:
    P = w.T * w.M + w.T * (w.T + 1) / 2
    return 4.0 * w.d * P * w.B * w.Hq


def traffic_for(kernel: str, workload: str):
    """HBM bytes per launch (FETCH_SIZE + WRITE_SIZE, copy-calibrated) from the
    committed rocprofv3 counter summary, or None if there is none or the
    kernel's sources changed since the counters were taken."""
    from paper_2608_19920_amd.counters import KERNELS, src_hash
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f).get(f"{kernel}@{workload}")
    if not rec or rec.get("src_hash") != src_hash(KERNELS[kernel][1]):
        return None
    return rec.get("bytes_per_launch")


# ----------------------------------------------------------------- device side
PREFILL_WARMUP = 3
PREFILL_REPS = 20


def interleaved_median_ms(fns, reps, warmup, torch):
    """Median duration in ms of each call in ``fns`` (name -> callable): after
    ``warmup`` untimed rounds, ``reps`` rounds that run the calls one after
    the other, each bracketed by a pair of events on the current stream, so
    every call is timed under the same conditions as the others."""
    for _ in range(warmup):
        for fn in fns.values():
            fn()
    torch.cuda.synchronize()
    E = lambda: torch.cuda.Event(enable_timing=True)
    ev = {k: [(E(), E()) for _ in range(reps)] for k in fns}
    for r in range(reps):
        for k, fn in fns.items():
            a, b = ev[k][r]
            a.record()
            fn()
            b.record()
    torch.cuda.synchronize()
    return {k: float(np.median([a.elapsed_time(b) for a, b in ev[k]])) for k in fns}


def _dev_state(x, torch):
    bf = torch.bfloat16
    to = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a)).to("cuda").to(dt)
    return dict(k_cache=to(x["k_cache"], bf), v_cache=to(x["v_cache"], bf),
                scores=to(x["scores"], torch.float32),
                token_pos=to(x["token_pos"], torch.int32))


def graph_steps(steps: int, avail: int) -> int:
    """Token steps per captured graph: the largest divisor of the timed step
    count that is at most 16 and at most the token steps the workload draws,
    so that the timed region is exactly `steps` token steps."""
    return max(g for g in range(1, min(16, avail, steps) + 1) if steps % g == 0)


def bench_decode(args, torch, H, W):
    w = W.WORKLOADS["decode_bf16"]
    bf = torch.bfloat16
    layers = []
    for layer in range(LAYERS):
        x = W.make_inputs(w, seed=layer)
        st = _dev_state(x, torch)
        to = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to("cuda").to(bf)
        # the workload's token steps: each its own query, new key and value
        inp = dict(q=[to(a) for a in x["q_steps"]], k_new=[to(a) for a in x["k_new_steps"]],
                   v_new=[to(a) for a in x["v_new_steps"]], pos0=int(x["pos0"]),
                   scale=float(x["scale"]))
        bufs = H.alloc_step(w.B, w.Hq, w.Hkv, w.T, w.M, w.d, bf)
        layers.append((st, inp, bufs))
    del x
    n_avail = len(layers[0][1]["q"])
    gsteps = graph_steps(args.steps, n_avail)

    def step(s):
        """Token step s (mod the drawn steps) over the layer states, in order."""
        s %= n_avail
        for st, inp, bufs in layers:
            H.step(st, inp["q"][s], inp["k_new"][s], inp["v_new"][s], bufs, inp["pos0"] + s,
                   inp["scale"])

    stream = torch.cuda.Stream()
    torch.cuda.synchronize()
    with torch.cuda.stream(stream):
        for s in range(args.warmup):             # eager warm-up on the capture stream
            step(s)
    torch.cuda.synchronize()
    # `gsteps` consecutive token steps x LAYERS layer states in one graph
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=stream):
        for s in range(gsteps):
            step(s)
    torch.cuda.synchronize()
    graph.replay()                               # untimed: the graph's first launch
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t_wall = time.perf_counter()
    e0.record()
    for _ in range(args.steps // gsteps):
        graph.replay()
    e1.record()
    torch.cuda.synchronize()
    t_wall = time.perf_counter() - t_wall
    ms_step = e0.elapsed_time(e1) / args.steps

    # Per-kernel durations: the same steps once more, eager, with the library
    # bracketing each of its launches by events on the launch stream.
    H.h2o_debug_timing(True)
    for s in range(args.steps):
        step(s)
    torch.cuda.synchronize()
    ktimes = {k: H.h2o_debug_kernel_time(k) for k in ("decode_split", "decode_finish")}
    H.h2o_debug_timing(False)
    step_bytes = decode_step_bytes(w) * LAYERS
    gbs = step_bytes / (ms_step * 1e-3) / 1e9

    # The same token step on ONE layer state, captured LAYERS times in a row:
    # its 69 MB stay in the 256 MB Infinity Cache between steps (hot MALL).
    st0, inp0, bufs0 = layers[0]
    hot = torch.cuda.CUDAGraph()
    with torch.cuda.graph(hot, stream=stream):
        for _ in range(LAYERS):
            H.step(st0, inp0["q"][0], inp0["k_new"][0], inp0["v_new"][0], bufs0, inp0["pos0"],
                   inp0["scale"])
    torch.cuda.synchronize()
    for _ in range(args.warmup):
        hot.replay()
    torch.cuda.synchronize()
    e0.record()
    for _ in range(args.steps):
        hot.replay()
    e1.record()
    torch.cuda.synchronize()
    hot_us = e0.elapsed_time(e1) / args.steps / LAYERS * 1e3
    hot_mall = {"workload": "the same token step on one layer state, replayed (its 69 MB "
                            "stay in the 256 MB Infinity Cache)",
                "us_per_layer_step": round(hot_us, 2),
                "gbs": round(decode_step_bytes(w) / (hot_us * 1e-6) / 1e9, 1)}
    ms_split, n_split = ktimes["decode_split"]
    avg_split_ms = ms_split / max(n_split, 1)
    ach = decode_split_bytes(w) / (avg_split_ms * 1e-3) / 1e9
    roof = {"kernel": "decode_split", "bound": "hbm", "achieved": round(ach, 1),
            "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(ach / HBM_PEAK_GBS, 4),
            "traffic": traffic_for("decode_split", w.name),
            "algorithmic_bytes_per_launch": decode_split_bytes(w),
            "avg_launch_us": round(avg_split_ms * 1e3, 2),
            "kernel_us": {k: round(v[0] / max(v[1], 1) * 1e3, 2) for k, v in ktimes.items()},
            "timing": "start/stop HIP events of hipExtLaunchKernel (stamped at the kernel's "
                      "own begin and end) on the launch stream, over an eager pass of the "
                      "timed steps"}
    return dict(w=w, ms_step=ms_step, value=gbs, roofline=roof, wall_s=t_wall,
                step_bytes=step_bytes, hot_mall=hot_mall, graph_steps=gsteps)


def bench_prefill(name, args, torch, H, W):
    w = W.WORKLOADS[name]
    x = W.make_inputs(w, seed=0)
    bf = torch.bfloat16
    to = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to("cuda").to(bf)
    st = _dev_state(x, torch)
    q, kn, vn = to(x["q"]), to(x["k_new"]), to(x["v_new"])
    pos0, scale = int(x["pos0"]), float(x["scale"])
    del x
    bufs = H.alloc_step(w.B, w.Hq, w.Hkv, w.T, w.M, w.d, bf)
    sdpa = lambda: H.h2o_sdpa_chunk(q, st["k_cache"], st["v_cache"], kn, vn, bufs["out"],
                                    bufs["lse"], bufs["wsum"], bufs["workspace"], scale)
    full = lambda: H.step(st, q, kn, vn, bufs, pos0, scale)
    # the attention call and the whole step (attention, accumulate, evict and
    # insert), interleaved, median of PREFILL_REPS after PREFILL_WARMUP
    med = interleaved_median_ms({"sdpa": sdpa, "full_step": full}, PREFILL_REPS,
                                PREFILL_WARMUP, torch)
    ms, ms_step = med["sdpa"], med["full_step"]
    # per-kernel durations of the same calls from the library's timing hook
    H.h2o_debug_timing(True)
    for _ in range(PREFILL_REPS):
        full()
    torch.cuda.synchronize()
    kt = {k: H.h2o_debug_kernel_time(k) for k in
          ("mfma_lse", "mfma_main", "split_reduce", "colsum_reduce", "accumulate", "bottomk",
           "insert", "bottomk_insert")}
    H.h2o_debug_timing(False)
    Wf = attention_flops(w)
    tf = Wf / (ms * 1e-3) / 1e12
    main_ms = kt["mfma_main"][0] / max(kt["mfma_main"][1], 1)
    ach_main = Wf / (main_ms * 1e-3) / 1e12
    return {"workload": w.describe(), "tflops": round(tf, 1),
            "frac_of_bf16_peak": round(tf / BF16_PEAK_TFLOPS, 4),
            "ms_sdpa": round(ms, 4), "ms_full_step": round(ms_step, 4),
            "timing": f"median of {PREFILL_REPS} after {PREFILL_WARMUP} warm-up rounds, "
                      "the two calls interleaved",
            "kernel_us": {k: round(v[0] / max(v[1], 1) * 1e3, 1) for k, v in kt.items()},
            "roofline_main": {"kernel": "mfma_main", "bound": "mfma",
                              "achieved": round(ach_main, 1), "peak": BF16_PEAK_TFLOPS,
                              "unit": "TFLOP/s", "frac": round(ach_main / BF16_PEAK_TFLOPS, 4),
                              "traffic": traffic_for("mfma_main", w.name)}}


# --------------------------------------------- the paper's order: insert first
def insert_first_flops(w) -> float:
    """Attention work of h2o_sdpa_cache after the chunk is in the cache: the
    M - T older slots are seen by all T queries, chunk key i by queries >= i."""
    P = (w.M - w.T) * w.T + w.T * (w.T + 1) / 2
    return 4.0 * w.d * P * w.B * w.Hq


def insert_first_step_bytes(w) -> int:
    """Algorithmic HBM bytes of one insert-first token step (T = 1)."""
    return decode_step_bytes(w) + w.B * w.Hkv * w.M * 4     # + the token positions read


def bench_insert_first(args, torch, H, W):
    """h2o_chunk_step_insert_first on the decode workload (8 layer states,
    consecutive token steps in one HIP graph, as in bench_decode) and
    h2o_sdpa_cache / the whole insert-first step on the prefill workloads."""
    bf = torch.bfloat16
    w = W.WORKLOADS["decode_bf16"]
    layers = []
    for layer in range(LAYERS):
        x = W.make_inputs(w, seed=layer)
        st = _dev_state(x, torch)
        to = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to("cuda").to(bf)
        inp = ([to(a) for a in x["q_steps"]], [to(a) for a in x["k_new_steps"]],
               [to(a) for a in x["v_new_steps"]], int(x["pos0"]), float(x["scale"]))
        layers.append((st, inp, H.alloc_step(w.B, w.Hq, w.Hkv, w.T, w.M, w.d, bf,
                                             insert_first=True)))
    del x
    n_avail = len(layers[0][1][0])
    gsteps = graph_steps(args.steps, n_avail)

    def step(s):
        s %= n_avail
        for st, (q, kn, vn, pos0, scale), b in layers:
            H.h2o_chunk_step_insert_first(q[s], st["k_cache"], st["v_cache"], st["scores"],
                                          st["token_pos"], kn[s], vn[s], b["out"], b["lse"],
                                          b["wsum"], b["evict_idx"], b["workspace"], pos0 + s,
                                          scale)

    stream = torch.cuda.Stream()
    torch.cuda.synchronize()
    with torch.cuda.stream(stream):
        for s in range(args.warmup):
            step(s)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=stream):
        for s in range(gsteps):
            step(s)
    torch.cuda.synchronize()
    graph.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(args.steps // gsteps):
        graph.replay()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    gbs = insert_first_step_bytes(w) * LAYERS / (ms * 1e-3) / 1e9
    out = {"decode": {"workload": w.describe() + f", {LAYERS} layer states",
                      "us_per_step": round(ms * 1e3, 1), "gbs": round(gbs, 1),
                      "frac_of_hbm_peak": round(gbs / HBM_PEAK_GBS, 4)},
           "prefill": []}
    del layers, graph
    torch.cuda.empty_cache()
    for name in PREFILL:
        w = W.WORKLOADS[name]
        x = W.make_inputs(w, seed=0)
        st = _dev_state(x, torch)
        to = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to("cuda").to(bf)
        q, kn, vn = to(x["q"]), to(x["k_new"]), to(x["v_new"])
        pos0, scale = int(x["pos0"]), float(x["scale"])
        del x
        b = H.alloc_step(w.B, w.Hq, w.Hkv, w.T, w.M, w.d, bf, insert_first=True)
        full = lambda: H.h2o_chunk_step_insert_first(
            q, st["k_cache"], st["v_cache"], st["scores"], st["token_pos"], kn, vn, b["out"],
            b["lse"], b["wsum"], b["evict_idx"], b["workspace"], pos0, scale)
        sdpa = lambda: H.h2o_sdpa_cache(q, st["k_cache"], st["v_cache"], st["token_pos"],
                                        b["out"], b["lse"], b["wsum"], b["workspace"], pos0,
                                        scale)
        full()                     # the chunk is in the cache from here on
        res = interleaved_median_ms({"sdpa_cache": sdpa, "full_step": full}, PREFILL_REPS,
                                    PREFILL_WARMUP, torch)
        tf = insert_first_flops(w) / (res["sdpa_cache"] * 1e-3) / 1e12
        out["prefill"].append({"workload": w.describe(), "tflops": round(tf, 1),
                               "frac_of_bf16_peak": round(tf / BF16_PEAK_TFLOPS, 4),
                               "ms_sdpa_cache": round(res["sdpa_cache"], 4),
                               "ms_full_step": round(res["full_step"], 4)})
        del st, q, kn, vn, b
        torch.cuda.empty_cache()
    return out


# ----------------------------------------------------------------- backward
def bench_backward(args, torch, H, W):
    """h2o_sdpa_chunk_backward on the first prefill workload, after its
    forward: TFLOP/s of the algorithmic backward work 2.5 W (the five
    products QK^T, dout V^T, P^T dout, dS K, dS^T Q over the visible pairs)."""
    w = W.WORKLOADS["prefill_bf16"]
    bf = torch.bfloat16
    x = W.make_inputs(w, seed=0)
    to = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to("cuda").to(bf)
    q, kc, vc, kn, vn = (to(x[n]) for n in ("q", "k_cache", "v_cache", "k_new", "v_new"))
    scale = float(x["scale"])
    del x
    b = H.alloc_step(w.B, w.Hq, w.Hkv, w.T, w.M, w.d, bf)
    H.h2o_sdpa_chunk(q, kc, vc, kn, vn, b["out"], b["lse"], b["wsum"], b["workspace"], scale)
    dout = torch.randn_like(q)
    grads = [torch.empty_like(t) for t in (q, kc, vc, kn, vn)]
    ws = torch.empty(max(H.h2o_backward_workspace_bytes(w.B, w.Hq, w.Hkv, w.T, w.M, w.d, bf), 16),
                     dtype=torch.uint8, device="cuda")
    fn = lambda: H.h2o_sdpa_chunk_backward(q, kc, vc, kn, vn, b["lse"], dout, *grads, ws, scale)
    reps = PREFILL_REPS
    ms = interleaved_median_ms({"bwd": fn}, reps, PREFILL_WARMUP, torch)["bwd"]
    # per-kernel times from the library's timing hook, over the same calls
    H.h2o_debug_timing(True)
    for _ in range(reps):
        fn()
    torch.cuda.synchronize()
    kern = {k: round(H.h2o_debug_kernel_time(k)[0] / reps * 1e3, 1)
            for k in ("bwd_dot", "bwd_dq", "bwd_dq_reduce", "bwd_dkdv")}
    H.h2o_debug_timing(False)
    tf = 2.5 * attention_flops(w) / (ms * 1e-3) / 1e12
    return {"workload": w.describe(), "ms": round(ms, 3), "tflops": round(tf, 1),
            "frac_of_bf16_peak": round(tf / BF16_PEAK_TFLOPS, 4), "kernel_us": kern,
            "kernels": "bf16 MFMA: rows pass for D, rows pass for dq (+ split reduce), "
                       "keys pass for dk/dv"}


# -------------------------------------------------------------- CPU baseline
def bench_variants(args, torch, H, W):
    """Eviction and insert under the paper's three score rankings (Sec.
    "Variants of Heavy-Hitter Oracle"): h2o_evict_insert_policy with
    h2o, h2o_norm (score over age) and h2o_orig (score summed over the batch,
    one slot set per KV head) on the chunked-prefill shapes, interleaved,
    median of PREFILL_REPS after PREFILL_WARMUP rounds. Each call evicts and
    inserts for real; the position advances by T per call so that every
    slot's age stays positive."""
    bf = torch.bfloat16
    out = []
    for name in PREFILL:
        w = W.WORKLOADS[name]
        x = W.make_inputs(w, seed=0)
        st = _dev_state(x, torch)
        to = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to("cuda").to(bf)
        kn, vn = to(x["k_new"]), to(x["v_new"])
        pos = [int(x["pos0"])]
        del x
        bufs = H.alloc_step(w.B, w.Hq, w.Hkv, w.T, w.M, w.d, bf)
        bufs["wsum"].uniform_(0.0, 1.0)
        fns = {}
        for policy in ("h2o", "h2o_norm", "h2o_orig"):
            ws = torch.empty(max(H.h2o_evict_workspace_bytes(w.B, w.Hkv, w.M, w.T, policy), 16),
                             dtype=torch.uint8, device="cuda")

            def fn(policy=policy, ws=ws):
                H.h2o_evict_insert_policy(st["k_cache"], st["v_cache"], st["scores"],
                                          st["token_pos"], kn, vn, bufs["wsum"],
                                          bufs["evict_idx"], pos[0], policy, ws)
                pos[0] += w.T
            fns[policy] = fn
        med = interleaved_median_ms(fns, PREFILL_REPS, PREFILL_WARMUP, torch)
        out.append({"workload": w.describe(), "k": w.T,
                    "us": {k: round(v * 1e3, 1) for k, v in med.items()}})
        del st, kn, vn, bufs
        torch.cuda.empty_cache()
    return out


def cpu_baseline(w, budget_s, W):
    import oracle
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count()
    x = W.make_inputs(w, seed=0)
    state = (x["k_cache"], x["v_cache"], x["scores"], x["token_pos"])
    n, t0 = 0, time.perf_counter()
    while True:
        s = n % w.steps
        r = oracle.h2o_step(*state, x["q_steps"][s], x["k_new_steps"][s], x["v_new_steps"][s],
                            int(x["pos0"]) + n, x["scale"])
        state = (r["k_cache"], r["v_cache"], r["scores"], r["token_pos"])
        n += 1
        if time.perf_counter() - t0 > budget_s or n >= 64:
            break
    dt = (time.perf_counter() - t0) / n
    return {"value": round(decode_step_bytes(w) / dt / 1e9, 4), "unit": "GB/s",
            "cores": int(threads), "kind": "oracle",
            "sample": f"{n} token steps of one layer state ({w.describe()}), float64 numpy",
            "s_per_step": round(dt, 3)}


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawTextHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--cpu-budget", type=float, default=15.0,
                    help="seconds of oracle work for the CPU baseline (0 = skip)")
    ap.add_argument("--no-prefill", action="store_true")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py: the benchmark runs on one GPU only; use --gpus 1", file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2608_19920_amd import h2o as H
    from paper_2608_19920_amd import workloads as W
    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        sys.exit(1)
    H.lib()
    print(f"# bench: decode {LAYERS} layer states, steps {args.steps}", file=sys.stderr, flush=True)
    dec = bench_decode(args, torch, H, W)
    print(f"# decode: {dec['ms_step']*1e3:.1f} us/step, {dec['value']:.0f} GB/s", file=sys.stderr,
          flush=True)
    prefill = []
    if not args.no_prefill:
        for name in PREFILL:
            r = bench_prefill(name, args, torch, H, W)
            print(f"# {name}: {r['tflops']} TFLOP/s", file=sys.stderr, flush=True)
            prefill.append(r)
            torch.cuda.empty_cache()
    ins = None
    if not args.no_prefill:
        ins = bench_insert_first(args, torch, H, W)
        print(f"# insert-first decode: {ins['decode']['gbs']} GB/s; prefill "
              f"{[r['tflops'] for r in ins['prefill']]} TFLOP/s", file=sys.stderr, flush=True)
    variants = None
    if not args.no_prefill:
        variants = bench_variants(args, torch, H, W)
        print(f"# evict+insert by policy (us): {[v['us'] for v in variants]}", file=sys.stderr,
              flush=True)
    bwd = None
    if not args.no_prefill:
        bwd = bench_backward(args, torch, H, W)
        print(f"# backward {bwd['workload']}: {bwd['ms']} ms, {bwd['tflops']} TFLOP/s",
              file=sys.stderr, flush=True)
    w = dec["w"]
    cpu = None
    if args.cpu_budget > 0:
        cpu = cpu_baseline(w, args.cpu_budget, W)
        print(f"# cpu oracle: {cpu['value']} GB/s on {cpu['cores']} threads", file=sys.stderr,
              flush=True)
    rec = {
        "metric": METRIC, "value": round(dec["value"], 1), "unit": "GB/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(dec["ms_step"], 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"decode_bf16 token step over {LAYERS} layer states "
                               f"(hipGraphs of {dec['graph_steps']} token steps, replayed)",
                   "B": w.B, "Hq": w.Hq, "Hkv": w.Hkv,
                   "d": w.d, "M": w.M, "T": w.T, "layers": LAYERS,
                   "bytes_per_step": dec["step_bytes"],
                   "frac_of_hbm_peak": round(dec["value"] / HBM_PEAK_GBS, 4)},
        "roofline": dec["roofline"],
        "hot_mall": dec["hot_mall"],
        "cpu_baseline": cpu,
        "prefill": prefill,
        "insert_first": ins,
        "variants": variants,
        "backward": bwd,
    }
    print(json.dumps(rec))


if __name__ == "__main__":
    main()
