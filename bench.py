"""Benchmark of one hybrid-batch decoder-layer iteration on one MI355X.

A step is one hb_run_iteration over the Llama-3-8B-shaped layer with one
512-token prefill chunk (offset drawn from 0..4096) plus 64 decodes (contexts
512..4096) over a 2M-token paged KV cache, inputs already resident in HBM.
Prints one JSON line: new tokens/s, per-step latency, the roofline of the
dominant kernel, the CPU oracle's rate on the same batch and the latency
profile against chunk size that dynamic chunking consumes.

    python bench.py [--gpus 1] [--steps 200] [--warmup 20]
"""
from __future__ import annotations

import argparse
import hashlib
import re
import json
import os
import subprocess
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM = 8.0e12       # MI355X HBM3E bytes/s
PEAK_BF16 = 2.5e15      # MI355X dense bf16 MFMA flop/s
RIDGE = PEAK_BF16 / PEAK_HBM
SETTLE_MS = 150.0       # continuous iterations before the measured passes


def log(msg: str) -> None:
    print(msg, file=sys.stderr, flush=True)


def kernel_work(shape, requests, out_f32=True):
    """Algorithmic (flops, HBM bytes) of each kernel for one iteration: the
    layer's algorithmic work (layer_work) split over the kernels that must do
    it. Bytes are what the method must move -- bf16 weights once, the cached
    and new K/V read once per (request, kv head), the new K/V written, x_in
    (bf16) and y -- and nothing an implementation adds: the intermediates q,
    the attention output, h2, the normed activations and the SwiGLU product
    are not counted. Flops: 2 T N K per GEMM, 4 n_q hd per unmasked (query,
    key) pair for attention, 4 T H per RMSNorm."""
    T = sum(c for c, _ in requests)
    H, nq, nkv, hd, F = shape.hidden, shape.n_q_heads, shape.n_kv_heads, shape.head_dim, shape.ffn_dim
    qd, qkv_n = nq * hd, (nq + 2 * nkv) * hd
    pairs = sum(c * x + c * (c + 1) / 2 for c, x in requests)
    kv_tok = sum(c + x for c, x in requests)
    kv_b = 2.0 * 2 * nkv * hd  # bf16 K and V of one token
    yb = 4 if out_f32 else 2
    return {
        "rmsnorm_attn": (4.0 * T * H, 2.0 * T * H + 2.0 * H),                 # x_in, g_attn
        # QKV projection with RoPE and the paged K/V scatter in its epilogue
        "gemm_qkv": (2.0 * T * H * qkv_n, 2.0 * H * qkv_n + kv_b * T),        # W_qkv, new K/V written
        "attention": (4.0 * nq * hd * pairs, kv_b * kv_tok),                   # cached + new K/V read
        "attn_merge": (0.0, 0.0),
        "gemm_o": (2.0 * T * qd * H, 2.0 * H * qd),                            # W_o
        "rmsnorm_ffn": (4.0 * T * H, 2.0 * H),                                 # g_ffn
        "gemm_gate_up": (2.0 * T * H * 2 * F, 2.0 * 2 * F * H),               # W_gate_up
        "gemm_down": (2.0 * T * F * H, 2.0 * H * F + yb * T * H),             # W_down, y
    }


def roofline_time_s(work):
    """Sum over kernels of max(flops / bf16 peak, bytes / HBM peak)."""
    return sum(max(f / PEAK_BF16, b / PEAK_HBM) for f, b in work.values())


def layer_work(shape, requests, out_f32=True):
    T = sum(c for c, _ in requests)
    H, nq, nkv, hd, F = shape.hidden, shape.n_q_heads, shape.n_kv_heads, shape.head_dim, shape.ffn_dim
    p_lin = shape.linear_params
    pairs = sum(c * x + c * (c + 1) / 2 for c, x in requests)
    kv_tok = sum(c + x for c, x in requests)
    flops = 2.0 * T * p_lin + 4.0 * nq * hd * pairs
    bytes_ = 2.0 * p_lin + 4.0 * H + 2.0 * 2 * nkv * hd * (kv_tok + T) + 2.0 * T * H + (4 if out_f32 else 2) * T * H
    return flops, bytes_


def kernel_sources_digest(names):
    """Digest of the code of the given sources: comments and whitespace are
    dropped, so that only a change to the code itself invalidates counters
    taken from it."""
    h = hashlib.sha256()
    for n in names:
        with open(os.path.join(ROOT, "paper_2503_22562_amd", "csrc", n)) as f:
            text = f.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(" ".join(text.split()).encode())
    return h.hexdigest()[:16]


TRAFFIC_SOURCES = {
    "attention": ["k_attention.hip", "hb_device.h", "hb_plan.h"],
    "gemm_gate_up": ["k_gemm.hip", "hb_device.h"],
    "gemm_down": ["k_gemm.hip", "hb_device.h"],
    "gemm_qkv": ["k_gemm.hip", "hb_device.h"],
    "gemm_o": ["k_gemm.hip", "hb_device.h"],
}


def measured_traffic(kernel, workload):
    """HBM bytes per launch from the committed rocprofv3 counter summary
    (profiles/traffic_<kernel>_<workload>.txt, `key: value` lines), only if the
    kernel's sources are unchanged since the counters were taken."""
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel}_{workload}.txt")
    if not os.path.exists(path) or kernel not in TRAFFIC_SOURCES:
        return None
    rec = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.startswith((" ", "#", "|")):
                k, v = line.split(":", 1)
                rec[k.strip()] = v.strip()
    if rec.get("sources_digest") != kernel_sources_digest(TRAFFIC_SOURCES[kernel]):
        return None
    try:
        return float(rec["bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def time_oracle(batch, weights_bits, min_cpu_s, max_wall_s, max_runs=None, w64=None):
    """Run the oracle (fp64 NumPy) on a batch repeatedly until min_cpu_s of
    oracle time (or max_wall_s of wall time, or max_runs runs) has passed;
    seeding each run's cached context is not timed. Returns the per-run
    seconds."""
    import oracle
    shape = batch.shape
    w64 = oracle.weights_to_f64(weights_bits) if w64 is None else w64
    x = oracle.bf16_bits_to_f64(batch.x_in())
    prior = {r: tuple(oracle.bf16_bits_to_f64(a) for a in batch.prior_kv(r))
             for r, q in enumerate(batch.requests) if q.context_len}
    times = []
    t_start = time.perf_counter()
    while True:
        cache = oracle.PagedKVCache(batch.num_blocks, shape.n_kv_heads, shape.head_dim)
        for r, (k, v) in prior.items():
            cache.write(batch.requests[r].block_table, 0, k, v)
        t0 = time.perf_counter()
        oracle.layer_forward(w64, shape, cache, batch.requests, x)
        times.append(time.perf_counter() - t0)
        if (sum(times) >= min_cpu_s or time.perf_counter() - t_start > max_wall_s
                or (max_runs and len(times) >= max_runs)):
            break
    return times


def blas_threads():
    threads = int(os.environ.get("OMP_NUM_THREADS", "0")) or os.cpu_count()
    try:
        from threadpoolctl import threadpool_info
        threads = max(int(i.get("num_threads", 0)) for i in threadpool_info()) or threads
    except Exception:
        pass
    return threads


def cpu_baseline(batch, weights_bits, min_cpu_s=10.0, max_wall_s=40.0):
    """The oracle (fp64 NumPy) on the same batch, on the host's cores, timed
    (repeated until min_cpu_s of oracle time), and once more on one thread."""
    import oracle
    w64 = oracle.weights_to_f64(weights_bits)
    times = time_oracle(batch, weights_bits, min_cpu_s, max_wall_s, w64=w64)
    one = None
    try:
        from threadpoolctl import threadpool_limits
        with threadpool_limits(limits=1):
            t1 = time_oracle(batch, weights_bits, 0.0, max_wall_s, max_runs=1, w64=w64)
        one = {"value": batch.n_tokens / t1[0], "unit": "tokens/s", "cores": 1, "seconds": round(t1[0], 2)}
    except Exception:
        pass
    total = float(sum(times))
    return {"value": batch.n_tokens * len(times) / total, "unit": "tokens/s", "cores": blas_threads(),
            "kind": "oracle", "cpu_model": cpu_model(), "one_thread": one,
            "sample": f"the bench batch ({batch.n_tokens} tokens, {len(batch.requests)} requests) run "
                      f"{len(times)} times, {total:.1f} s of fp64 NumPy oracle time (cached-context seeding not "
                      f"timed); one_thread: one more run on a single BLAS thread"}


def cpu_baselines():
    """The oracle on the host's cores over the configurations of the layer's
    workloads (one JSON line per configuration, then a summary line): the
    tiny layer, the 8B bench batch (also on one thread), the 8B multi-request
    batch, the sweep's corner cells (chunk 128 / 2048 x 0 / 256 decodes), the
    70B layer (one run). Median of 3 runs, except the 70B layer. A reported
    baseline of the oracle as it stands, not a target."""
    from threadpoolctl import threadpool_limits
    from hb_workloads import (LLAMA3_70B, LLAMA3_8B, TINY, llama70b_batch, llama8b_batch, make_weights, multi_batch,
                              sweep_batch, tiny_batch)
    import oracle
    cases = [("tiny: chunk 64 at 128 + 8 decodes at 256", TINY, tiny_batch, 3, None),
             ("llama3-8b: chunk 512 + 64 decodes (bench batch)", LLAMA3_8B, llama8b_batch, 3, None),
             ("llama3-8b: chunk 512 + 64 decodes (bench batch), one thread", LLAMA3_8B, llama8b_batch, 1, 1),
             ("llama3-8b: 4 chunks + 256 decodes", LLAMA3_8B, multi_batch, 3, None)]
    for c in (128, 2048):
        for n in (0, 256):
            cases.append((f"llama3-8b sweep: chunk {c} + {n} decodes", LLAMA3_8B,
                          (lambda c=c, n=n: sweep_batch(c, n)), 3, None))
    cases.append(("llama3-70b: chunk 2048 at 30720 + 32 decodes at 32768", LLAMA3_70B, llama70b_batch, 1, None))
    weights = {}
    out = []
    for name, shape, mk, runs, threads in cases:
        if shape.name not in weights:
            weights.clear()
            weights[shape.name] = oracle.weights_to_f64(make_weights(shape))
        b = mk()
        log(f"cpu baseline: {name}")
        if threads:
            with threadpool_limits(limits=threads):
                t = time_oracle(b, None, 1e30, 1e30, max_runs=runs, w64=weights[shape.name])
        else:
            t = time_oracle(b, None, 1e30, 1e30, max_runs=runs, w64=weights[shape.name])
        fl, _ = layer_work(shape, [(q.chunk_len, q.context_len) for q in b.requests])
        med = float(np.median(t))
        rec = {"config": name, "tokens": b.n_tokens, "requests": len(b.requests), "runs": len(t),
               "median_s": round(med, 3), "tokens_per_s": round(b.n_tokens / med, 1),
               "gflops": round(fl / med / 1e9, 1), "threads": threads or blas_threads()}
        print(json.dumps(rec), flush=True)
        out.append(rec)
    print(json.dumps({"cpu_model": cpu_model(), "nproc": os.cpu_count(),
                      "affinity": len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else None,
                      "blas_threads": blas_threads(), "oracle": "fp64 NumPy (oracle/layer.py)",
                      "configs": out}), flush=True)
    return 0


def copy_calibration(nbytes=1 << 30, reps=3):
    """A plain device copy of known size: nbytes read and nbytes written per
    launch. Profiling it with the same counters as the kernels gives the
    factor between what FETCH_SIZE / WRITE_SIZE report and the bytes moved."""
    import torch
    torch.cuda.set_device(0)
    a = torch.empty(nbytes, dtype=torch.uint8, device="cuda").fill_(1)
    b = torch.empty_like(a)
    torch.cuda.synchronize()
    for _ in range(reps):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": nbytes, "launches": reps}), flush=True)
    return 0


def counters_cell(cell, steps, warmup):
    """Only the layer iterations of one gate cell, for counter passes
    (rocprofv3 --pmc): 'C,D' = the 8B sweep cell with a C-token chunk and D
    decodes, '70b' = the 70B layer's chunk 2048 at 30720 + 32 decodes,
    'multi' = the 8B 4-chunk + 256-decode batch, '8b' = the bench batch."""
    import torch
    from hb_workloads import LLAMA3_8B, LLAMA3_70B, llama70b_batch, llama8b_batch, multi_batch, sweep_batch
    from paper_2503_22562_amd import hb
    from paper_2503_22562_amd.harness import to_device_bf16
    torch.cuda.set_device(0)
    if cell == "70b":
        shape, b = LLAMA3_70B, llama70b_batch()
    elif cell == "multi":
        shape, b = LLAMA3_8B, multi_batch()
    elif cell == "8b":
        shape, b = LLAMA3_8B, llama8b_batch()
    else:
        c, d = (int(v) for v in cell.split(","))
        shape, b = LLAMA3_8B, sweep_batch(c, d)
    layer = DeviceRandomLayer(hb, torch, shape, b.num_blocks, b.n_tokens, max(len(b.requests), 1), 7)
    reqs = [(q.chunk_len, q.context_len, q.block_table) for q in b.requests]
    x = to_device_bf16(b.x_in())
    y = torch.empty((b.n_tokens, shape.hidden), dtype=torch.float32, device="cuda")
    for _ in range(warmup + steps):
        layer.run(reqs, x, hb.HB_OUT_F32, y)
    torch.cuda.synchronize()
    print(json.dumps({"counters_cell": cell, "tokens": b.n_tokens, "iterations": warmup + steps}), flush=True)
    return 0


def regime(hb, dl, batch, shape, x_dev, y_dev, steps):
    """Per-kernel timing of one sweep cell: every launch bracketed by HIP
    events, the cell run `steps` times after two warm-up iterations."""
    reqs = [(q.chunk_len, q.context_len, q.block_table) for q in batch.requests]
    for _ in range(2):
        dl.run(reqs, x_dev, hb.HB_OUT_F32, y_dev)
    hb.hb_set_kernel_timing(dl.layer, True)
    hb.hb_kernel_times(dl.layer, reset=True)
    for _ in range(steps):
        dl.run(reqs, x_dev, hb.HB_OUT_F32, y_dev)
    times = hb.hb_kernel_times(dl.layer, reset=True)
    hb.hb_set_kernel_timing(dl.layer, False)
    work = kernel_work(shape, [(c, xx) for c, xx, _ in reqs])
    out = {}
    for name, (tot, n) in times.items():
        if n:
            fl, by = work.get(name, (0.0, 0.0))
            out[name] = (tot / n * 1e-3, fl, by)
    return out


def fit_and_validate_latency_model(hb, dl, shape, mixes, median_ms, iters):
    """Fit the iteration latency model (hb_fit_latency_model) to the latency
    profile's cells plus cells whose chunk follows a 4096-token context, then
    time batches off that grid with hb_profile_batches (the same kernel-only,
    cold-cache timing) against the model's predictions, and let the chunk
    selector pick chunks for three slacks next to 64 decodes."""
    import torch
    from hb_workloads import (SWEEP_CHUNKS, llama8b_batch, make_batch, multi_batch, sweep_batch,
                              sweep_decode_contexts)
    from paper_2503_22562_amd.harness import to_device_bf16
    extra = [([], 4096), (sweep_decode_contexts(64), 4096)]
    prof2 = hb.hb_profile(dl.layer, SWEEP_CHUNKS, extra, warmup=3, iters=iters, seed=2)
    model = hb.hb_fit_latency_model(dl.cfg, SWEEP_CHUNKS, list(mixes) + extra,
                                    np.vstack([median_ms, prof2["median_ms"]]))
    rng = np.random.default_rng(21)

    def timed(batches):
        keep, args = [], []
        for b in batches:
            x = to_device_bf16(b.x_in())
            y = torch.empty((b.n_tokens, shape.hidden), dtype=torch.float32, device="cuda")
            keep.append((x, y))
            args.append(([(q.chunk_len, q.context_len, q.block_table) for q in b.requests], x, y))
        return hb.hb_profile_batches(dl.layer, args, warmup=3, iters=iters)["median_ms"]

    vals = {"chunk 512 at 3431 + 64 decodes (the bench batch)": llama8b_batch(),
            "4 chunks + 256 decodes (multi-request batch)": multi_batch(),
            "chunk 384 + 64 decodes": sweep_batch(384, 64),
            "200 decodes, contexts U{256..8192}": make_batch(shape, [(1, int(c)) for c in rng.integers(256, 8192, 200)], 41),
            "chunk 768 at 6000 + 100 decodes": make_batch(
                shape, [(768, 6000)] + [(1, int(c)) for c in rng.integers(512, 4096, 100)], 42),
            "chunk 2048 at 8192": make_batch(shape, [(2048, 8192)], 43)}
    meas = timed(vals.values())
    validation = []
    for (name, b), m in zip(vals.items(), meas):
        p = hb.hb_predict_latency(model, dl.cfg, [(q.chunk_len, q.context_len) for q in b.requests])
        validation.append({"batch": name, "measured_ms": round(float(m), 4), "predicted_ms": round(p, 4)})
    errs = [abs(v["predicted_ms"] / v["measured_ms"] - 1) for v in validation]
    ctx = [int(c) for c in rng.integers(512, 4096, 64)]
    picks, sel_batches = [], []
    margin = model.fit_max_under
    for slack in (0.45, 0.6, 0.9):
        c, p = hb.hb_select_chunk(model, dl.cfg, ctx, [100.0 + slack] * 64, 100.0, 2048, 4096, 32, margin)
        picks.append((slack, c, p))
        sel_batches.append(make_batch(shape, [(max(c, 1), 2048)] + [(1, x) for x in ctx], 50))
    sel_meas = timed(sel_batches)
    return {"features": ["1", "T/1e3", "KV GB read", "attention TFLOP vs cached context",
                         "attention TFLOP within new tokens"],
            "coef_ms": [round(c, 5) for c in model.coef], "fit_cells": model.n_cells,
            "fit_rel_rms": round(model.fit_rel_rms, 4), "fit_max_under": round(model.fit_max_under, 4),
            "selector_margin": round(margin, 4), "validation": validation,
            "validation_mape": round(float(np.mean(errs)), 4), "validation_max_err": round(float(np.max(errs)), 4),
            "selector": [{"decodes": 64, "chunk_context": 2048, "slack_ms": s, "chunk": c,
                          "predicted_ms": round(p, 4), "measured_ms": round(float(m), 4)}
                         for (s, c, p), m in zip(picks, sel_meas)],
            "timing": "kernel time per iteration, 512 MiB written and another 512 MiB read before each (hb_profile / hb_profile_batches)"}


class DeviceRandomLayer:
    """A layer whose weights and paged pool are drawn on the device from a
    seed (for timing only: values need realistic scale, not the oracle's
    exact draws); exposes .layer and .run like the harness's DeviceLayer."""

    def __init__(self, hb, torch, shape, num_blocks, max_T, max_R, seed):
        self.hb, self.torch = hb, torch
        g = torch.Generator(device="cuda")
        g.manual_seed(seed)
        self.w = random_layer_weights(torch, shape, g)
        nkv, hd = shape.n_kv_heads, shape.head_dim
        self.k = torch.randn((num_blocks, nkv, 16, hd), generator=g, device="cuda", dtype=torch.bfloat16)
        self.v = torch.randn((num_blocks, nkv, 2, hd, 8), generator=g, device="cuda", dtype=torch.bfloat16)
        self.layer = hb.hb_create_layer(hb.make_config(shape, max_T, max_R), self.w, self.k, self.v, num_blocks)

    def run(self, reqs, x, out_dtype, y):
        self.hb.hb_run_iteration(self.layer, reqs, x, y, out_dtype)
        return y


def random_layer_weights(torch, shape, g):
    H, F, nq, nkv, hd = shape.hidden, shape.ffn_dim, shape.n_q_heads, shape.n_kv_heads, shape.head_dim

    def randn(rows, cols, std):
        return (torch.randn((rows, cols), generator=g, device="cuda") * std).to(torch.bfloat16)

    return {"w_qkv": randn((nq + 2 * nkv) * hd, H, H ** -0.5), "w_o": randn(H, nq * hd, (nq * hd) ** -0.5),
            "w_gate_up": randn(2 * F, H, H ** -0.5), "w_down": randn(H, F, F ** -0.5),
            "g_attn": (1 + 0.1 * torch.randn(H, generator=g, device="cuda")).to(torch.bfloat16),
            "g_ffn": (1 + 0.1 * torch.randn(H, generator=g, device="cuda")).to(torch.bfloat16)}


def blas_ceiling(torch, shape, M, steps=10):
    """Context only: torch.matmul (hipBLASLt) on the layer's four GEMM shapes
    at M rows, no epilogues (microseconds, TFLOP/s)."""
    H, F, qd, qkv_n = shape.hidden, shape.ffn_dim, shape.n_q_heads * shape.head_dim, \
        (shape.n_q_heads + 2 * shape.n_kv_heads) * shape.head_dim
    out = {}
    for name, N, K in (("gemm_qkv", qkv_n, H), ("gemm_o", H, qd), ("gemm_gate_up", 2 * F, H), ("gemm_down", H, F)):
        a = torch.randn((M, K), device="cuda").to(torch.bfloat16)
        w = torch.randn((N, K), device="cuda").to(torch.bfloat16)
        for _ in range(3):
            c = a @ w.t()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(steps):
            c = a @ w.t()
        e1.record()
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) / steps * 1e3
        out[name] = {"us": round(us, 1), "tflops": round(2.0 * M * N * K / us / 1e6, 1),
                     "weight_tb_s": round(2.0 * N * K / us / 1e6, 2)}
        del a, w, c
    tot_us = sum(v["us"] for v in out.values())
    shapes = ((qkv_n, H), (H, qd), (2 * F, H), (H, F))
    tot_fl = sum(2.0 * M * N * K for N, K in shapes)
    out["four_gemms"] = {"us": round(tot_us, 1), "mfma_frac": round(tot_fl / (tot_us * 1e-6) / PEAK_BF16, 4),
                         "weight_tb_s": round(sum(2.0 * N * K for N, K in shapes) / tot_us / 1e6, 2)}
    return out


def regime_cell(hb, torch, layer, b, shp, steps, rates=None):
    """One batch on a layer, every launch bracketed by events: attention's
    HBM and MFMA fractions, the four GEMMs' MFMA fraction (split-K reduces
    included) and weight rate, per-GEMM TFLOP/s."""
    from paper_2503_22562_amd.harness import to_device_bf16
    x = to_device_bf16(b.x_in())
    y = torch.empty((b.n_tokens, shp.hidden), dtype=torch.float32, device="cuda")
    kt = regime(hb, layer, b, shp, x, y, steps)
    at_s, at_f, at_b = kt["attention"]
    gem = {k: v for k, v in kt.items() if k.startswith("gemm_")}
    g_s = sum(t for t, _, _ in gem.values())
    g_f = sum(f for _, f, _ in gem.values())
    w_bytes = 2.0 * shp.hidden * ((shp.n_q_heads + 2 * shp.n_kv_heads) * shp.head_dim
                                  + shp.n_q_heads * shp.head_dim + 3 * shp.ffn_dim)
    return {"layer_ms": round(sum(t for t, _, _ in kt.values()) * 1e3, 4),
            "attention_ms": round(at_s * 1e3, 4), "attention_hbm_frac": round(at_b / at_s / PEAK_HBM, 4),
            "attention_mfma_frac": round(at_f / at_s / PEAK_BF16, 4),
            "gemms_ms": round(g_s * 1e3, 4), "gemms_mfma_frac": round(g_f / g_s / PEAK_BF16, 4),
            "gemms_weight_tb_s": round(w_bytes / g_s / 1e12, 2),
            "per_gemm_tflops": {k: round(f / t / 1e12, 1) for k, (t, f, _) in sorted(gem.items())},
            **({"attention_frac_of_sustained_read": round(at_b / at_s / (rates["random_4kb_read_tb_s"] * 1e12), 4),
                "gemms_frac_of_sustained_mfma": round(g_f / g_s / (rates["mfma_bf16_pflop_s"] * 1e15), 4)}
               if rates else {})}


def gate_cells(hb, torch, dl, shape, steps, with_70b=True, rates=None):
    """The fixed gate sets of the layer's targets: attention's HBM fraction on
    decode-heavy sweep cells (chunk 128/256 x 128/256 decodes), the four
    GEMMs' MFMA fraction on chunk-heavy cells (chunk 1024/2048 x 0/32 decodes)
    and on the 70B layer (chunk 2048 at 30720 + 32 decodes at 32768); with
    hipBLASLt on the same GEMM shapes as context."""
    from hb_workloads import LLAMA3_70B, llama70b_batch, sweep_batch

    def cell(layer, b, shp):
        return regime_cell(hb, torch, layer, b, shp, steps, rates)

    out = {"decode_heavy": {}, "chunk_heavy": {}}
    for c in (128, 256):
        for n in (128, 256):
            out["decode_heavy"][f"chunk {c} + {n} decodes"] = cell(dl, sweep_batch(c, n), shape)
    for c in (1024, 2048):
        for n in (0, 32):
            out["chunk_heavy"][f"chunk {c} + {n} decodes"] = cell(dl, sweep_batch(c, n), shape)
    for m in (256, 576, 2048):
        out[f"blas_ceiling_8b_m{m}"] = blas_ceiling(torch, shape, m)
    if with_70b:
        b70 = llama70b_batch()
        l70 = DeviceRandomLayer(hb, torch, LLAMA3_70B, b70.num_blocks, b70.n_tokens, 64, 170)
        out["chunk_heavy"]["llama3-70b: chunk 2048 at 30720 + 32 decodes at 32768"] = cell(l70, b70, LLAMA3_70B)
        del l70
        torch.cuda.empty_cache()
        out["blas_ceiling_70b_m2080"] = blas_ceiling(torch, LLAMA3_70B, 2080)
    dh = [v["attention_hbm_frac"] for v in out["decode_heavy"].values()]
    ch = [v["gemms_mfma_frac"] for v in out["chunk_heavy"].values()]
    out["summary"] = {"decode_heavy_attention_hbm_frac_min": min(dh), "target_hbm": 0.60,
                      "chunk_heavy_gemms_mfma_frac_min": min(ch), "chunk_heavy_gemms_mfma_frac_max": max(ch),
                      "target_mfma": 0.50}
    if rates:
        out["summary"]["decode_heavy_attention_frac_of_sustained_read_min"] = min(
            v["attention_frac_of_sustained_read"] for v in out["decode_heavy"].values())
        out["summary"]["chunk_heavy_gemms_frac_of_sustained_mfma_min"] = min(
            v["gemms_frac_of_sustained_mfma"] for v in out["chunk_heavy"].values())
    return out


def tp_shard_cells(hb, torch, steps, rates=None):
    """One GPU's share of a layer under tensor parallelism, sharded by heads
    (the 8B layer at TP2 on the bench batch's request mix, the 70B layer at
    TP8 on the 70B mix): the shard's kernels at their real shapes, timed like
    the gate cells. The two all-reduces of the [T, hidden] activations per
    layer that tensor parallelism adds are not run on one GPU; their bf16
    payload is reported."""
    from hb_workloads import LLAMA3_8B_TP2, LLAMA3_70B_TP8, llama70b_batch, llama8b_batch
    out = {}
    for shp, b in ((LLAMA3_8B_TP2, llama8b_batch(shape=LLAMA3_8B_TP2)),
                   (LLAMA3_70B_TP8, llama70b_batch(shape=LLAMA3_70B_TP8))):
        layer = DeviceRandomLayer(hb, torch, shp, b.num_blocks, b.n_tokens, len(b.requests), shp.weight_seed)
        c = regime_cell(hb, torch, layer, b, shp, steps, rates)
        c["shape"] = {"hidden": shp.hidden, "n_q_heads": shp.n_q_heads, "n_kv_heads": shp.n_kv_heads,
                      "head_dim": shp.head_dim, "ffn_dim": shp.ffn_dim}
        c["tokens"] = b.n_tokens
        c["allreduce_bytes_per_layer"] = 2 * b.n_tokens * shp.hidden * 2
        out[b.label] = c
        del layer
        torch.cuda.empty_cache()
    return out


def model_iteration(hb, torch, shape, batch_lens, seed, n_layers=32, vocab=128256, steps=20, warmup=3):
    """Whole-model iteration (hb_run_model): n_layers decoder layers of the
    given shape between a token embedding and the LM head, on the same
    request mix as the layer bench. Weights and cached K/V are drawn on the
    device (seeded; they only need realistic sizes and finite values here);
    each layer has its own pool, sized to the blocks the batch uses."""
    from hb_workloads import make_batch
    need = sum(-(-(c + x) // 16) for c, x in batch_lens)
    nb = need + 64
    b = make_batch(shape, batch_lens, seed, num_blocks=nb)
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    H, F, nq, nkv, hd = shape.hidden, shape.ffn_dim, shape.n_q_heads, shape.n_kv_heads, shape.head_dim

    layers, pools = [], []
    for _ in range(n_layers):
        layers.append(random_layer_weights(torch, shape, g))
        pools.append((torch.randn((nb, nkv, 16, hd), generator=g, device="cuda", dtype=torch.bfloat16),
                      torch.randn((nb, nkv, 2, hd, 8), generator=g, device="cuda", dtype=torch.bfloat16)))
    embed = torch.randn((vocab, H), generator=g, device="cuda", dtype=torch.bfloat16)
    head = (torch.randn((vocab, H), generator=g, device="cuda") * H ** -0.5).to(torch.bfloat16)
    g_final = (1 + 0.1 * torch.randn(H, generator=g, device="cuda")).to(torch.bfloat16)
    cfg = hb.make_config(shape, max(b.n_tokens, 1), max(len(b.requests), 1))
    model = hb.hb_create_model(cfg, layers, pools, nb, embed, g_final, head)
    reqs = [(q.chunk_len, q.context_len, q.block_table) for q in b.requests]
    ids = torch.from_numpy(b.token_ids(vocab)).to("cuda")
    nxt = torch.empty(len(reqs), dtype=torch.int32, device="cuda")
    for _ in range(warmup):
        hb.hb_run_model(model, reqs, ids, nxt)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    for i in range(steps):
        ev[i][0].record(stream)
        hb.hb_run_model(model, reqs, ids, nxt)
        ev[i][1].record(stream)
    torch.cuda.synchronize()
    ts = sorted(s.elapsed_time(e) for s, e in ev)
    med = ts[len(ts) // 2]
    T = b.n_tokens
    weight_gb = (n_layers * (H * (nq + 2 * nkv) * hd + nq * hd * H + 3 * H * F) + vocab * H) * 2 / 1e9
    del model, layers, pools, embed, head
    torch.cuda.empty_cache()
    return {"layers": n_layers, "vocab": vocab, "tokens": T, "requests": len(reqs),
            "median_ms": round(med, 4), "p10_ms": round(ts[len(ts) // 10], 4),
            "p90_ms": round(ts[(9 * len(ts)) // 10], 4), "tokens_per_s": round(T / (med * 1e-3), 1),
            "weights_gb": round(weight_gb, 2),
            "note": "time between tokens of every decode in the batch = one iteration; "
                    "compare with the strictest QoS tier's 50 ms"}


def gpu_max_clock_mhz():
    """The first GPU agent's maximum shader clock as rocminfo reports it (None
    if rocminfo is unavailable)."""
    try:
        out = subprocess.run(["rocminfo"], capture_output=True, text=True, timeout=30).stdout
    except (OSError, subprocess.SubprocessError):
        return None
    gpu = False
    for line in out.splitlines():
        if "Device Type:" in line:
            gpu = "GPU" in line
        elif gpu and "Max Clock Freq. (MHz):" in line:
            try:
                return int(line.split(":")[1].split()[0])
            except (IndexError, ValueError):
                return None
    return None


def device_rates(hb, torch, gib=8):
    """Sustained rates of this GPU on fixed patterns (hb_measure_device_rates
    over a gib-GiB region, about the paged pool's size): random 4-KB-chunk
    reads (the paged-attention pattern), a streaming read, bf16 MFMAs on
    varied operands. Context for the roofline fractions, whose denominators
    stay the published peaks."""
    buf = torch.empty(gib << 30, dtype=torch.uint8, device="cuda")
    r = hb.hb_measure_device_rates(buf)
    del buf
    torch.cuda.empty_cache()
    return {"random_4kb_read_tb_s": round(r["random_4kb_read_bytes_per_s"] / 1e12, 3),
            "stream_read_tb_s": round(r["stream_read_bytes_per_s"] / 1e12, 3),
            "mfma_bf16_pflop_s": round(r["mfma_bf16_flop_per_s"] / 1e15, 3), "region_gib": gib}


def device_info(torch):
    p = torch.cuda.get_device_properties(0)
    return {"name": p.name, "arch": getattr(p, "gcnArchName", None), "compute_units": p.multi_processor_count,
            "max_clock_mhz": gpu_max_clock_mhz(), "hbm_gib": round(p.total_memory / 2 ** 30, 1),
            "host_cores": len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count()}


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-profile", action="store_true")
    ap.add_argument("--profile-iters", type=int, default=100)
    ap.add_argument("--profile-warmup", type=int, default=10)
    ap.add_argument("--regime-steps", type=int, default=10)
    ap.add_argument("--no-regimes", action="store_true")
    ap.add_argument("--no-model", action="store_true", help="skip the 32-layer whole-model iteration")
    ap.add_argument("--counters-cell", default=None,
                    help="only run one cell ('C,D', '70b', 'multi' or '8b') --warmup + --steps times (counter passes) and exit")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 1 GiB device copy (counter calibration) and exit")
    ap.add_argument("--cpu-baselines", action="store_true",
                    help="only time the CPU oracle over the workload configurations (no GPU) and exit")
    a = ap.parse_args()
    if a.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the hybrid-batch layer runs on a single MI355X; "
              "run it with --gpus 1.", file=sys.stderr)
        return 2
    if a.copy_calibration:
        return copy_calibration()
    if a.cpu_baselines:
        return cpu_baselines()
    if a.counters_cell:
        return counters_cell(a.counters_cell, a.steps, a.warmup)

    import torch
    from hb_workloads import LLAMA3_8B, POOL_TOKENS, SWEEP_CHUNKS, SWEEP_DECODES, llama8b_batch, make_weights, \
        sweep_decode_contexts
    from paper_2503_22562_amd import hb
    from paper_2503_22562_amd.harness import DeviceLayer, to_device_bf16

    torch.cuda.set_device(0)
    shape = LLAMA3_8B
    batch = llama8b_batch()
    reqs = [(q.chunk_len, q.context_len, q.block_table) for q in batch.requests]
    T = batch.n_tokens
    log(f"bench: {batch.label}, T={T}; generating weights and cached context")
    w = make_weights(shape)
    dl = DeviceLayer(shape, w, POOL_TOKENS // 16, 4096, 512, pool_fill_bits=0)
    for r, q in enumerate(batch.requests):
        if q.context_len:
            k, v = batch.prior_kv(r)
            dl.append_kv(q.block_table, 0, k, v)
    x = to_device_bf16(batch.x_in())
    y = torch.empty((T, shape.hidden), dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()

    log(f"bench: warmup {a.warmup}")
    for _ in range(a.warmup):
        dl.run(reqs, x, hb.HB_OUT_F32, y)
    torch.cuda.synchronize()

    work = kernel_work(shape, [(c, xx) for c, xx, _ in reqs])

    # The GPU runs its first tens of milliseconds of work after an idle spell
    # at lower clocks (about 40 ms of iterations to reach steady state on
    # MI355X). Steady serving keeps it busy, so the measured passes start
    # after SETTLE_MS of continuous iterations, with no host gap longer than
    # a synchronisation before the timed region.
    n_settle = max(a.steps, int(np.ceil(SETTLE_MS / 0.4)))
    for _ in range(n_settle):
        dl.run(reqs, x, hb.HB_OUT_F32, y)
    # per-kernel breakdown (every launch bracketed by events) picks the dominant kernel
    n_breakdown = max(a.steps, 50)
    hb.hb_set_kernel_timing(dl.layer, True)
    for _ in range(n_breakdown):
        dl.run(reqs, x, hb.HB_OUT_F32, y)
    breakdown = hb.hb_kernel_times(dl.layer, reset=True)
    kernels = {}
    for name, (tot, n) in breakdown.items():
        if n == 0:
            continue
        avg_ms = tot / n
        fl, by = work.get(name, (0.0, 0.0))
        kernels[name] = {"avg_ms": round(avg_ms, 5), "launches": n,
                         "tflops": round(fl / (avg_ms * 1e-3) / 1e12, 2) if fl else None,
                         "gbps": round(by / (avg_ms * 1e-3) / 1e9, 1) if by else None,
                         "roofline_frac": round(max(fl / PEAK_BF16, by / PEAK_HBM) / (avg_ms * 1e-3), 4)}
    dom = max(kernels, key=lambda k: kernels[k]["avg_ms"] * kernels[k]["launches"])

    # timed region: W warm-up iterations, then exactly `steps` iterations;
    # HIP events on the layer's stream bracket only the dominant kernel's
    # launches (two event records per step)
    hb.hb_set_kernel_timing(dl.layer, [dom])
    for _ in range(a.warmup):
        dl.run(reqs, x, hb.HB_OUT_F32, y)
    hb.hb_kernel_times(dl.layer, reset=True)  # synchronises; drops the warm-up's events
    t0 = time.perf_counter()
    for _ in range(a.steps):
        dl.run(reqs, x, hb.HB_OUT_F32, y)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    dom_ms, dom_n = hb.hb_kernel_times(dl.layer, reset=True)[dom]
    hb.hb_set_kernel_timing(dl.layer, False)
    ms_per_step = wall * 1e3 / a.steps
    log(f"bench: {ms_per_step:.4f} ms/step")

    # same iteration without any events, and with the Infinity Cache flushed
    # before each: 512 MiB written, then another 512 MiB read, so that the
    # written lines are evicted (and written back) before the timed iteration
    flush = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    flush_w, flush_r = flush[:512 << 20], flush[512 << 20:]
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(a.steps)]
    for i in range(a.steps):
        flush_w.fill_(i & 0xFF)
        flush_r.max()
        ev[i][0].record(stream)
        dl.run(reqs, x, hb.HB_OUT_F32, y)
        ev[i][1].record(stream)
    torch.cuda.synchronize()
    cold = sorted(s.elapsed_time(e) for s, e in ev)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    for _ in range(a.steps):
        dl.run(reqs, x, hb.HB_OUT_F32, y)
    torch.cuda.synchronize()
    plain_ms = (time.perf_counter() - t1) * 1e3 / a.steps
    del flush

    fl, by = work[dom]
    avg_s = dom_ms / dom_n * 1e-3
    if fl / by > RIDGE:
        roof = {"bound": "mfma", "achieved": round(fl / avg_s / 1e12, 2), "peak": PEAK_BF16 / 1e12,
                "unit": "TFLOP/s"}
    else:
        roof = {"bound": "hbm", "achieved": round(by / avg_s / 1e9, 1), "peak": PEAK_HBM / 1e9, "unit": "GB/s"}
    roof["frac"] = round(roof["achieved"] / roof["peak"], 4)
    roof["kernel"] = dom
    roof["avg_ms"] = round(dom_ms / dom_n, 5)
    roof["launches_timed"] = dom_n
    roof["algorithmic_flops"] = fl
    roof["algorithmic_bytes"] = by
    tr = measured_traffic(dom, "llama3-8b")
    roof["traffic"] = tr
    log("bench: device rates (random 4-KB reads, streaming read, MFMA loop)")
    rates = device_rates(hb, torch)
    sus = rates["mfma_bf16_pflop_s"] * 1e3 if roof["bound"] == "mfma" else rates["random_4kb_read_tb_s"] * 1e3
    roof["sustained_peak"] = round(sus, 1)
    roof["frac_of_sustained"] = round(roof["achieved"] / sus, 4) if sus > 0 else None
    roof["sustained_note"] = ("sustained_peak: this GPU's rate measured in this run on the kernel's pattern "
                              "(bf16 MFMA loop on varied operands, or random 4-KB reads for an HBM-bound "
                              "kernel; device.rates); context only, frac uses the published peak")
    flops, bytes_ = layer_work(shape, [(c, xx) for c, xx, _ in reqs])
    step_s = ms_per_step * 1e-3

    # the gate cells of the layer's targets (decode-heavy: attention's HBM
    # rate; chunk-heavy: the GEMMs' MFMA rate), hipBLASLt as context
    gates = shards = None
    if not a.no_regimes:
        log("bench: gate cells (decode-heavy and chunk-heavy sweep cells, 70B layer, hipBLASLt ceiling)")
        gates = gate_cells(hb, torch, dl, shape, a.regime_steps, rates=rates)
        log("bench: tensor-parallel shards (8B at TP2, 70B at TP8)")
        shards = tp_shard_cells(hb, torch, a.regime_steps, rates=rates)

    profile = None
    if not a.no_profile:
        log("bench: latency profile (chunk x decode grid)")
        mixes = [(sweep_decode_contexts(n), 0) for n in SWEEP_DECODES]
        prof = hb.hb_profile(dl.layer, SWEEP_CHUNKS, mixes, warmup=a.profile_warmup, iters=a.profile_iters, seed=1)
        med = prof["median_ms"]
        mono = all(med[i, j] * (1.01 if (n == 0 and SWEEP_CHUNKS[j] <= 256) else 1.0) >= med[i, j - 1]
                   for i, n in enumerate(SWEEP_DECODES) for j in range(1, len(SWEEP_CHUNKS)))
        profile = {"chunks": list(SWEEP_CHUNKS), "decodes": list(SWEEP_DECODES),
                   "median_ms": np.round(med, 4).tolist(), "p90_ms": np.round(prof["p90_ms"], 4).tolist(),
                   "tokens_per_s": np.round(prof["tokens_per_s"]).tolist(),
                   "hbm_frac": np.round(prof["hbm_frac"], 3).tolist(),
                   "mfma_frac": np.round(prof["mfma_frac"], 3).tolist(),
                   "monotone_in_chunk": bool(mono), "cache": "before each timed iteration 512 MiB written, then another 512 MiB read",
                   "iterations_per_cell": {"warmup": a.profile_warmup, "timed": a.profile_iters}}

    latency_model = None
    if not a.no_profile:
        log("bench: latency model (fit, off-grid validation, chunk selection)")
        latency_model = fit_and_validate_latency_model(hb, dl, shape, mixes, prof["median_ms"], a.profile_iters)

    model = None
    if not a.no_model:
        log("bench: whole-model iteration (32 layers, LM head)")
        model = model_iteration(hb, torch, shape, [(c, xx) for c, xx, _ in reqs], batch.seed)

    cpu = None
    if not a.no_cpu_baseline:
        log("bench: CPU oracle baseline")
        del dl
        torch.cuda.empty_cache()
        cpu = cpu_baseline(batch, w)

    out = {
        "metric": "hybrid-batch layer throughput (new tokens/s) and latency",
        "value": round(T / step_s, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": a.steps,
        "warmup": a.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded random-init weights, N(0,1) activations and cached K/V)",
        "config": {"workload": "llama3-8b layer: 1 prefill chunk of 512 at offset U{0..4096} + 64 decodes, "
                               "contexts U{512..4096}, 2M-token paged pool", "tokens_per_step": T,
                   "requests": len(reqs), "hidden": shape.hidden, "q_heads": shape.n_q_heads,
                   "kv_heads": shape.n_kv_heads, "head_dim": shape.head_dim, "ffn": shape.ffn_dim,
                   "kv_block": 16, "parallelism": "none (1 GPU)"},
        "latency_ms": {"timed_region_per_step": round(ms_per_step, 5),
                       "no_events": round(plain_ms, 5),
                       "cache_flushed_median": round(cold[len(cold) // 2], 5),
                       "cache_flushed_p10": round(cold[len(cold) // 10], 5),
                       "cache_flushed_p90": round(cold[(9 * len(cold)) // 10], 5)},
        "layer_roofline": {"algorithmic_gflop": round(flops / 1e9, 2), "algorithmic_mb": round(bytes_ / 1e6, 1),
                           "mfma_frac": round(flops / step_s / PEAK_BF16, 4),
                           "hbm_frac": round(bytes_ / step_s / PEAK_HBM, 4),
                           "roofline_time_us": round(roofline_time_s(work) * 1e6, 1),
                           "frac": round(roofline_time_s(work) / step_s, 4),
                           "note": "roofline time = sum over kernels of max(flops / bf16 peak, bytes / HBM peak); "
                                   "frac = roofline time / ms_per_step"},
        "roofline": roof,
        "kernels": kernels,
        "kernels_note": "per-kernel averages from a separate pass with every launch bracketed by events; "
                        "bytes and flops are each kernel's share of the layer's algorithmic work",
        "passes": {"settle_steps": n_settle, "breakdown_steps": n_breakdown, "warmup": a.warmup,
                   "timed_steps": a.steps},
        "cpu_baseline": cpu,
        "gates": gates,
        "gates_note": "per-kernel averages with every launch bracketed by events; algorithmic work as for roofline; "
                      "GEMM times include their split-K reduces; gemms_weight_tb_s = the four GEMMs' weight bytes / "
                      "their time; blas_ceiling = torch.matmul (hipBLASLt) on the same shapes without epilogues, one "
                      "weight copy reused (context, not a target)",
        "tp_shards": shards,
        "tp_shards_note": "one GPU's share of a layer sharded by heads (QKV and gate/up by output columns, O and "
                          "down by input columns, pool and attention by kv head), timed as the gate cells; the two "
                          "all-reduces per layer that tensor parallelism adds are not run on one GPU "
                          "(allreduce_bytes_per_layer: their bf16 payload)",
        "latency_profile": profile,
        "latency_model": latency_model,
        "model_iteration": model,
        "device": dict(device_info(torch), rates=rates),
    }
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
