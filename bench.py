"""Benchmark: the 60 s, batch-64, 28-layer SpeechKV job on one MI355X.

One step is the whole hot path over one batch of synthetic input
(Qwen3-1.7B attention shapes: 16 query / 8 KV heads, head_dim 128; 32 prefix
tokens + 750 speech frames; layers 14..27 pooled with w = 4):
  prefill  28 x (pool the raw K/V into the paged cache, prefill attention of
           the 782 full-resolution queries over the compressed cache);
  decode   128 steps x 28 layers of one-query attention, each storing the new
           token's K/V in the cache.
The step is captured once as a HIP graph and replayed; inputs are resident in
HBM.  `value` is generated tokens per second of the whole job
(64 x 128 tokens per step).  The same job without compression (every layer at
full resolution) is measured beside it.

Also reported: the decode kernel's achieved HBM bandwidth against the 8 TB/s
peak (algorithmic bytes: every cached K/V row once, plus q, the new K/V and
the output) and against the attainable rate of a plain streaming read of the
same byte counts, measured in the same run; the pooling kernel's achieved HBM bandwidth (raw K/V read once,
cache rows written once) and the prefill attention's achieved bf16 TFLOP/s
against the 2.5 PFLOP/s dense MFMA peak (FLOPs of the visible (row, key) pairs
only), each from a graph of that kernel alone; HS Compression's pooling of
the whole hidden state (hidden 2048) on the same batch and spans, in GB/s;
the training backward of one layer (attention and pooling gradients) and the
prefill attention alone at the 1596-query prefill workload; decode over
10-minute audio at batch 16 (all 28 layers, w = 2, 4 and 8 against no
compression); and the fp64 CPU oracle timed on a bounded sample of the same
job.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu] [--no-full]
    python bench.py --traffic [--workload NAME]   # eager launches for counter runs
    python bench.py --traffic --train             # one training layer, eagerly
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "decode-attn achieved HBM GB/s & tokens/s/GPU, 60s audio b=64, pooled vs full KV"
HBM_PEAK_GBPS = 8000.0
BF16_MFMA_PEAK_TFLOPS = 2500.0  # dense


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def capture(fn):
    import torch
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        fn()  # one eager pass on the capture stream before capture
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        fn()
    torch.cuda.synchronize()
    return g


WARM_MS = 30.0  # untimed replays before a measurement: clocks ramp up over ~20 ms of load


def time_graph(g, reps, warm=None):
    """Average milliseconds per replay of graph g over `reps` replays, after
    untimed replays: `warm` of them, or by default as many as take WARM_MS
    (at least one; a short graph timed right after an idle gap otherwise
    reads up to 15% slow while the clocks ramp up)."""
    import torch
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    if warm is None:
        torch.cuda.synchronize()
        start.record()
        g.replay()
        end.record()
        torch.cuda.synchronize()
        once = max(start.elapsed_time(end), 1e-3)
        warm = min(int(WARM_MS / once), 1000)
    for _ in range(warm):
        g.replay()
    torch.cuda.synchronize()
    start.record()
    for _ in range(reps):
        g.replay()
    end.record()
    torch.cuda.synchronize()
    return start.elapsed_time(end) / reps  # ms


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "decode_kernel_stack60s_traffic.md")
DECODE_SOURCES = [os.path.join(ROOT, "paper_2607_06827_amd", "csrc", f)
                  for f in ("decode_attn.hip", "common.hpp", "kernels.hpp")]


def decode_source_hash():
    import hashlib
    h = hashlib.sha256()
    for f in DECODE_SOURCES:
        h.update(open(f, "rb").read())
    return h.hexdigest()[:16]


def measured_traffic():
    """HBM bytes per decode launch from the committed counter summary, or None
    when it is missing or was taken on a different decode kernel source."""
    try:
        text = open(TRAFFIC_FILE).read()
    except OSError:
        return None
    vals = dict(line.split(":", 1) for line in text.splitlines()
                if line.startswith(("traffic_bytes_per_launch:", "decode_source_sha256:")))
    if vals.get("decode_source_sha256", "").strip() != decode_source_hash():
        return None
    return float(vals["traffic_bytes_per_launch"])


def decode_launch_stats(job):
    """Algorithmic bytes and launch count of the decode part of one step."""
    total = sum(job.decode_bytes(s) for s in range(job.wl.decode_steps))
    launches = job.wl.decode_steps * len(job.layers)
    return total, launches


# (blocks, threads, loads in flight per buffer): the fastest of a sweep over
# 256..8192 blocks x 256..1024 threads x 1..8 loads at both launch sizes
STREAM_SHAPES = ((8192, 256, 1), (8192, 256, 2), (8192, 512, 1), (8192, 512, 2), (4096, 256, 2),
                 (4096, 512, 2), (1024, 1024, 4), (512, 512, 2))


def stream_ceiling(job, reps=3, copies=14):
    """Attainable HBM read rate for the decode launches of one step: a plain
    non-temporal streaming read of two buffers (bench-only kernel,
    libskv_bench.so) at the average K+V size of a pooled-layer and of a
    full-layer launch, best of a few launch shapes, rotating `copies` buffer
    pairs so the 256 MB last-level cache holds none of them.  Each launch of
    the step is then priced at its class's rate."""
    import ctypes
    import torch
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2607_06827_amd", "libskv_bench.so"))
    f = lib.skv_stream_read
    f.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int, ctypes.c_int,
                  ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
    f.restype = ctypes.c_int
    wl = job.wl
    classes = {}
    for i, l in enumerate(job.layers):
        key = "pooled" if l >= job.l0 else "full"
        classes.setdefault(key, []).extend(job.decode_bytes_layer(i, s) for s in range(wl.decode_steps))
    sink = torch.zeros(4, dtype=torch.int32, device="cuda")
    rates = {}
    for key, sizes in classes.items():
        half = int(sum(sizes) / len(sizes) / 2) // 1024 * 1024
        bufs = [(torch.empty(half, dtype=torch.uint8, device="cuda"),
                 torch.empty(half, dtype=torch.uint8, device="cuda")) for _ in range(copies)]
        best = 0.0
        for blocks, threads, depth in STREAM_SHAPES:
            def run():
                st = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
                for a, b in bufs:
                    rc = f(a.data_ptr(), b.data_ptr(), half, blocks, threads, depth, sink.data_ptr(), st)
                    if rc:
                        raise RuntimeError(f"skv_stream_read failed ({rc})")
            ms = time_graph(capture(run), reps) / copies
            best = max(best, 2 * half / (ms * 1e-3) / 1e9)
        rates[key] = best
        del bufs
        torch.cuda.empty_cache()
    total = sum(sum(v) for v in classes.values())
    seconds = sum(sum(v) / (rates[k] * 1e9) for k, v in classes.items())
    return {"gbps": total / seconds / 1e9,
            "pooled_launch_gbps": rates.get("pooled"), "full_launch_gbps": rates.get("full"),
            "probe": f"non-temporal streaming read of two buffers, best of {len(STREAM_SHAPES)} launch "
                     f"shapes, {copies} rotated buffer pairs"}


def measure(job, steps, warmup, label):
    g_step = capture(job.run)
    g_dec = capture(lambda: [job.run_decode_step(s) for s in range(job.wl.decode_steps)])
    g_pre = capture(job.run_prefill)
    g_pool = capture(job.run_pool)
    g_attn = capture(job.run_prefill_attn)
    wl = job.wl
    nl = len(job.layers)
    # the decode launches of each layer class on their own (same order and
    # cache contents as in the step)
    classes = {"pooled": [i for i, l in enumerate(job.layers) if l >= job.l0],
               "full": [i for i, l in enumerate(job.layers) if l < job.l0]}
    g_cls = {k: capture(lambda ix=ix: [job.decode_layer(i, s) for s in range(wl.decode_steps)
                                       for i in ix])
             for k, ix in classes.items() if ix}
    for _ in range(warmup):
        g_step.replay()
    ms_step = time_graph(g_step, steps, warm=0)  # (the W warmup steps ran above)
    ms_dec = time_graph(g_dec, max(2, steps))
    ms_pre = time_graph(g_pre, max(2, steps))
    ms_pool = time_graph(g_pool, max(2, steps))
    ms_attn = time_graph(g_attn, max(2, steps))
    dec_cls = {}
    for k, g in g_cls.items():
        ms = time_graph(g, max(2, steps))
        n = len(classes[k]) * wl.decode_steps
        nbytes = sum(job.decode_bytes_layer(i, s) for i in classes[k] for s in range(wl.decode_steps))
        dec_cls[k] = {"layers": len(classes[k]), "avg_launch_us": ms / n * 1e3,
                      "bytes_per_launch": nbytes / n,
                      "achieved_gbps": nbytes / (ms * 1e-3) / 1e9}
    del g_cls
    dec_bytes, launches = decode_launch_stats(job)
    pool_bytes = sum(job.pool_bytes_layer(i) for i in range(nl))
    attn_flops = sum(job.prefill_flops_layer(i) for i in range(nl))
    attn_bytes = sum(job.prefill_bytes_layer(i) for i in range(nl))
    res = {
        "ms_per_step": ms_step,
        "tokens_per_s": wl.batch * wl.decode_steps / (ms_step * 1e-3),
        "decode_ms": ms_dec,
        "decode_tokens_per_s": wl.batch * wl.decode_steps / (ms_dec * 1e-3),
        "decode_gbps": dec_bytes / (ms_dec * 1e-3) / 1e9,
        "decode_bytes_per_step": dec_bytes,
        "decode_launches": launches,
        "decode_classes": dec_cls,
        "prefill_ms": ms_pre,
        "pool": {"avg_launch_us": ms_pool / nl * 1e3,
                 "achieved_gbps": pool_bytes / (ms_pool * 1e-3) / 1e9,
                 "bytes_per_launch": pool_bytes / nl},
        "prefill_attn": {"avg_launch_us": ms_attn / nl * 1e3,
                         "achieved_tflops": attn_flops / (ms_attn * 1e-3) / 1e12,
                         "flops_per_launch": attn_flops / nl},
    }
    res["pool"]["frac_of_hbm_peak"] = res["pool"]["achieved_gbps"] / HBM_PEAK_GBPS
    res["prefill_attn"]["frac_of_bf16_mfma_peak"] = (res["prefill_attn"]["achieved_tflops"]
                                                     / BF16_MFMA_PEAK_TFLOPS)
    # roofline fraction: the larger of the MFMA and HBM floors over the measured time
    t_floor = max(attn_flops / (BF16_MFMA_PEAK_TFLOPS * 1e12), attn_bytes / (HBM_PEAK_GBPS * 1e9))
    res["prefill_attn"]["bytes_per_launch"] = attn_bytes / nl
    res["prefill_attn"]["roofline_frac"] = t_floor / (ms_attn * 1e-3)
    log(f"{label}: step {ms_step:.3f} ms, decode {ms_dec:.3f} ms "
        f"({res['decode_gbps']:.0f} GB/s), prefill+pool {ms_pre:.3f} ms "
        f"(pool {ms_pool:.3f} ms, {res['pool']['achieved_gbps']:.0f} GB/s; "
        f"attention {ms_attn:.3f} ms, {res['prefill_attn']['achieved_tflops']:.0f} TFLOP/s)")
    del g_step, g_dec, g_pre, g_pool, g_attn
    return res


def measure_adaptive(base, steps, warmup, num_splits):
    """The same step with a window that grows with depth (adaptive compression
    ratios across layers, future work in Sec. VI): each compressed layer pools
    and attends with its own window, so its cache has its own length."""
    from paper_2607_06827_amd import inputs
    from paper_2607_06827_amd.workload import Job

    wl = inputs.ADAPTIVE_W_60S
    job = Job(wl, share_inputs=base, num_splits=num_splits)
    g_step = capture(job.run)
    g_dec = capture(lambda: [job.run_decode_step(s) for s in range(wl.decode_steps)])
    for _ in range(warmup):
        g_step.replay()
    ms_step = time_graph(g_step, steps, warm=0)
    ms_dec = time_graph(g_dec, max(2, steps))
    dec_bytes, _ = decode_launch_stats(job)
    res = {"workload": wl.name, "w_layers": list(wl.w_layers[wl.l0:]), "ms_per_step": ms_step,
           "tokens_per_s": wl.batch * wl.decode_steps / (ms_step * 1e-3), "decode_ms": ms_dec,
           "decode_gbps": dec_bytes / (ms_dec * 1e-3) / 1e9,
           "cache_rows": [job.prefill_clen[i] for i in range(wl.l0, wl.num_layers)]}
    log(f"adaptive windows: step {ms_step:.3f} ms, decode {ms_dec:.3f} ms "
        f"({res['decode_gbps']:.0f} GB/s)")
    del g_step, g_dec, job
    return res


def measure_fused(base, steps, copies=4):
    """Pooling and prefill attention as one launch (pooling on the fly inside
    the attention, Sec. III-C) against the two launches: at the 1596-query
    workload (one layer, `copies` jobs in turn so that no launch finds its
    inputs in the last-level cache) and over the prefill of the whole stack."""
    from paper_2607_06827_amd import inputs
    from paper_2607_06827_amd.workload import Job

    wl = inputs.PREFILL_1500
    jobs = [Job(wl.with_(seed=wl.seed + i)) for i in range(copies)]
    g_split = capture(lambda: [j.run_prefill() for j in jobs])
    g_fused = capture(lambda: [j.run_prefill_fused() for j in jobs])
    us_split = time_graph(g_split, max(10, steps)) / copies * 1e3
    us_fused = time_graph(g_fused, max(10, steps)) / copies * 1e3
    del g_split, g_fused, jobs
    g_split = capture(base.run_prefill)
    g_fused = capture(base.run_prefill_fused)
    ms_split = time_graph(g_split, max(2, steps))
    ms_fused = time_graph(g_fused, max(2, steps))
    del g_split, g_fused
    log(f"fused pool+prefill ({wl.name}): {us_fused:.1f} us against {us_split:.1f} us as two "
        f"launches; stack prefill {ms_fused:.3f} ms against {ms_split:.3f} ms")
    return {"workload": wl.name, "fused_us": us_fused, "split_us": us_split,
            "fused_over_split": us_fused / us_split, "stack_workload": base.wl.name,
            "stack_prefill_fused_ms": ms_fused, "stack_prefill_split_ms": ms_split}


def measure_prefill_1596(steps, copies=4):
    """Prefill attention alone at the 1596-query x 471-key workload (b=8,
    16/8 heads): `copies` independent jobs, pooled once beforehand, run in
    turn so that no launch finds its 120 MB of inputs and outputs in the
    256 MB last-level cache."""
    from paper_2607_06827_amd import inputs
    from paper_2607_06827_amd.workload import Job

    wl = inputs.PREFILL_1500
    jobs = [Job(wl.with_(seed=wl.seed + i)) for i in range(copies)]
    for j in jobs:
        j.run_pool()
    g = capture(lambda: [j.run_prefill_attn() for j in jobs])
    ms = time_graph(g, max(10, steps)) / copies
    j = jobs[0]
    flops, nbytes = j.prefill_flops_layer(0), j.prefill_bytes_layer(0)
    t_floor = max(flops / (BF16_MFMA_PEAK_TFLOPS * 1e12), nbytes / (HBM_PEAK_GBPS * 1e9))
    tflops = flops / (ms * 1e-3) / 1e12
    log(f"prefill attention ({wl.name}, rotated): {ms * 1e3:.1f} us, {tflops:.0f} TFLOP/s, "
        f"roofline fraction {t_floor / (ms * 1e-3):.3f}")
    del g, jobs
    return {"workload": wl.name, "avg_launch_us": ms * 1e3, "flops_per_launch": flops,
            "bytes_per_launch": nbytes, "achieved_tflops": tflops,
            "frac_of_bf16_mfma_peak": tflops / BF16_MFMA_PEAK_TFLOPS,
            "achieved_gbps": nbytes / (ms * 1e-3) / 1e9,
            "floor_us": t_floor * 1e6, "roofline_frac": t_floor / (ms * 1e-3),
            "buffers": f"{copies} rotated jobs"}


def measure_segments(steps, copies=4):
    """Pooling + prefill attention of a multi-turn batch (three speech turns
    per sequence, segment tables) against a batch of the same rows and
    compressed length laid out as one run per sequence."""
    from paper_2607_06827_amd.workload import MULTI_TURN, SegmentJob

    res = {"segments": [list(x) for x in MULTI_TURN], "batch": 16}
    for name, one in (("segments_us", False), ("one_run_us", True)):
        jobs = [SegmentJob(MULTI_TURN, seed=6 + i, one_run=one) for i in range(copies)]
        g = capture(lambda: [j.run() for j in jobs])
        res[name] = time_graph(g, max(10, steps)) / copies * 1e3
        del g, jobs
    log(f"multi-turn pool+prefill (b=16, 1261 rows, 418 keys): {res['segments_us']:.1f} us with "
        f"segment tables, {res['one_run_us']:.1f} us as one run")
    return res


def measure_hs_pool(wl, steps, copies=4):
    """HS Compression's hidden-state pooling on the same batch and spans.

    One launch moves about 263 MB, close to the 256 MB of last-level cache
    (Infinity Cache): the graph runs `copies` independent jobs in turn so that
    no launch finds its input left in the cache by the one before."""
    from paper_2607_06827_amd.workload import HiddenPoolJob

    jobs = [HiddenPoolJob(wl.with_(seed=wl.seed + i)) for i in range(copies)]
    g = capture(lambda: [j.run() for j in jobs])
    ms = time_graph(g, max(10, steps)) / copies
    nbytes = jobs[0].bytes()
    gbps = nbytes / (ms * 1e-3) / 1e9
    log(f"hs pool (hidden {jobs[0].hidden}): {ms * 1e3:.1f} us, {gbps:.0f} GB/s")
    res = {"hidden": jobs[0].hidden, "avg_launch_us": ms * 1e3, "bytes_per_launch": nbytes,
           "achieved_gbps": gbps, "frac_of_hbm_peak": gbps / HBM_PEAK_GBPS}
    del g, jobs
    return res


def measure_long_sweep(steps, windows=(2, 4, 8)):
    """Decode over 10-minute audio (16 sequences, 32 + 7500 rows, 256 decode
    steps, all 28 layers) for each window w with layers 14..27 pooled, and
    the same job with no compression.  Raw K/V are generated once and shared;
    each configuration pools its caches, then its 256 x 28 decode launches
    are captured as one graph and timed.  The split count is the library's
    choice (split-K with a log-sum-exp merge where it pays)."""
    import torch
    from paper_2607_06827_amd import inputs
    from paper_2607_06827_amd.speechkv import speechkv_decode_num_splits
    from paper_2607_06827_amd.workload import Job

    wl = inputs.LONG_10MIN
    base = None
    res = {"workload": wl.name, "batch": wl.batch, "layers": wl.num_layers, "l0": wl.l0,
           "decode_steps": wl.decode_steps, "configs": {}}
    for w in (None,) + tuple(windows):
        name = "no_compression" if w is None else f"w{w}"
        job = Job(wl.with_(w=w or wl.w), l0=wl.num_layers if w is None else wl.l0,
                  with_prefill=False, share_inputs=base)
        if base is None:
            base = job
        job.run_prefill()
        g = capture(lambda: [job.run_decode_step(s) for s in range(wl.decode_steps)])
        ms = time_graph(g, max(2, steps // 2))
        del g
        total = sum(job.decode_bytes(s) for s in range(wl.decode_steps))
        pooled = [i for i, l in enumerate(job.layers) if l >= job.l0]
        full = [i for i, l in enumerate(job.layers) if l < job.l0]
        cfg = {"ms_per_decode_step": ms / wl.decode_steps,
               "gb_per_decode_step": total / wl.decode_steps / 1e9,
               "achieved_gbps": total / (ms * 1e-3) / 1e9,
               "frac_of_hbm_peak": total / (ms * 1e-3) / 1e9 / HBM_PEAK_GBPS,
               "tokens_per_s": wl.batch * wl.decode_steps / (ms * 1e-3),
               "cache_rows": {"pooled": job.prefill_clen[pooled[0]] if pooled else None,
                              "full": job.prefill_clen[full[0]] if full else None},
               "splits": {"pooled": speechkv_decode_num_splits(
                              wl.batch, wl.num_kv_heads, job.prefill_clen[pooled[0]] + wl.decode_steps)
                          if pooled else None,
                          "full": speechkv_decode_num_splits(
                              wl.batch, wl.num_kv_heads, job.prefill_clen[full[0]] + wl.decode_steps)
                          if full else None}}
        res["configs"][name] = cfg
        log(f"10-minute decode {name}: {cfg['ms_per_decode_step']:.3f} ms per step "
            f"({cfg['gb_per_decode_step']:.2f} GB, {cfg['achieved_gbps']:.0f} GB/s)")
        if job is not base:
            del job
        torch.cuda.empty_cache()
    full_ms = res["configs"]["no_compression"]["ms_per_decode_step"]
    for name, cfg in res["configs"].items():
        cfg["speedup_over_no_compression"] = full_ms / cfg["ms_per_decode_step"]
    del base
    torch.cuda.empty_cache()
    return res


def measure_train_bwd(steps, copies=4):
    """The training backward of one layer (Sec. III-C) at the 1596-query x
    471-key prefill workload: attention backward (dQ, dK^, dV^) and pooling
    backward (raw dK, dV and the gate's du).  `copies` independent jobs run in
    turn so that no launch finds its inputs left in the last-level cache."""
    from paper_2607_06827_amd import inputs
    from paper_2607_06827_amd.workload import TrainJob

    wl = inputs.PREFILL_1500
    jobs = [TrainJob(wl.with_(seed=wl.seed + i)) for i in range(copies)]
    for j in jobs:
        j.run_forward()
    g_attn = capture(lambda: [j.run_attn_bwd() for j in jobs])
    g_pool = capture(lambda: [j.run_pool_bwd() for j in jobs])
    ms_attn = time_graph(g_attn, max(10, steps)) / copies
    ms_pool = time_graph(g_pool, max(10, steps)) / copies
    j = jobs[0]
    flops, abytes, pbytes = j.attn_bwd_flops(), j.attn_bwd_bytes(), j.pool_bwd_bytes()
    tflops = flops / (ms_attn * 1e-3) / 1e12
    gbps = pbytes / (ms_pool * 1e-3) / 1e9
    t_floor = max(flops / (BF16_MFMA_PEAK_TFLOPS * 1e12), abytes / (HBM_PEAK_GBPS * 1e9))
    log(f"train backward ({wl.name}): attention {ms_attn * 1e3:.1f} us ({tflops:.0f} TFLOP/s), "
        f"pooling {ms_pool * 1e3:.1f} us ({gbps:.0f} GB/s)")
    res = {"workload": wl.name,
           "attn_bwd": {"avg_launch_us": ms_attn * 1e3, "flops_per_launch": flops,
                        "achieved_tflops": tflops, "frac_of_bf16_mfma_peak": tflops / BF16_MFMA_PEAK_TFLOPS,
                        "bytes_per_launch": abytes, "roofline_frac": t_floor / (ms_attn * 1e-3)},
           "pool_bwd": {"avg_launch_us": ms_pool * 1e3, "bytes_per_launch": pbytes,
                        "achieved_gbps": gbps, "frac_of_hbm_peak": gbps / HBM_PEAK_GBPS}}
    del g_attn, g_pool, jobs
    return res


def cpu_baseline(job, budget_s=15.0):
    """The fp64 oracle on whole sequences of the same job (all layers: pool,
    prefill attention, every decode step), one sequence at a time until about
    budget_s seconds of oracle time; tokens/s = decoded tokens / oracle time."""
    import numpy as np
    import torch
    import oracle

    wl = job.wl
    f64 = lambda t: t.detach().to("cpu", torch.float64).numpy()
    P, T, N = [wl.prefix_len], [wl.speech_len], [wl.suffix_len]
    spent, seqs = 0.0, 0
    for b in range(wl.batch):
        for i, l in enumerate(job.layers):
            k, v = f64(job.k_raw[i][b:b + 1]), f64(job.v_raw[i][b:b + 1])
            u, q = f64(job.gate[i]), f64(job.q_prefill[i][b:b + 1])
            qd = f64(job.q_dec[i][:, b])
            kn, vn = f64(job.k_new[i][:, b]), f64(job.v_new[i][:, b])
            t0 = time.perf_counter()
            kh, vh, clen = oracle.pool(k, v, P, T, N, wl.window(l), l, job.l0, u)
            oracle.attention(q, kh, vh, P, T, N, wl.window(l), l, job.l0, 0, job.scale)
            L = int(clen[0])
            K = np.concatenate([kh[:, :L], kn[None]], axis=1)
            V = np.concatenate([vh[:, :L], vn[None]], axis=1)
            for s in range(wl.decode_steps):
                oracle.decode(qd[s][None], K[:, :L + s + 1], V[:, :L + s + 1], [L + s + 1],
                              job.scale)
            spent += time.perf_counter() - t0
        seqs += 1
        if spent >= budget_s:
            break
    return {
        "value": seqs * wl.decode_steps / spent,
        "unit": "tokens/s",
        "cores": oracle.num_threads(),
        "cpu_model": cpu_model(),
        "kind": "oracle",
        "sample": (f"{seqs} of {wl.batch} sequences, whole job (28 layers: pool, prefill "
                   f"attention, {wl.decode_steps} decode steps), fp64, {spent:.1f} s"),
    }


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-full", action="store_true", help="skip the uncompressed run")
    ap.add_argument("--no-extras", action="store_true",
                    help="time the benchmark step only (no fused, multi-turn, adaptive-window, "
                         "HS-pooling or training figures), e.g. for a kernel trace of that step")
    ap.add_argument("--num-splits", type=int, default=0)
    ap.add_argument("--traffic", action="store_true",
                    help="counter-collection run: the job's launches and one HS pooling launch "
                         "issued eagerly once, then a plain 1 GiB device copy that calibrates the byte counters")
    ap.add_argument("--train", action="store_true",
                    help="with --traffic: one training layer of the 1596-query prefill workload "
                         "instead (forward, then attention and pooling backward)")
    ap.add_argument("--workload", default=None,
                    help="with --traffic: run this workload (by name) instead of the benchmark's")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}); the decode, "
              "pooling and prefill kernels run on a single device and nothing here shards "
              "across GPUs.", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2607_06827_amd import inputs
    from paper_2607_06827_amd.workload import Job

    wl = inputs.STACK_60S
    if args.train and not args.traffic:
        print("--train applies to --traffic runs only", file=sys.stderr)
        sys.exit(2)
    if args.workload:
        if not args.traffic:
            print("--workload applies to --traffic runs only", file=sys.stderr)
            sys.exit(2)
        named = {x.name: x for x in inputs.WORKLOADS}
        if args.workload not in named:
            print(f"unknown workload {args.workload}; one of {sorted(named)}", file=sys.stderr)
            sys.exit(2)
        wl = named[args.workload]
    torch.cuda.set_device(0)
    if args.train:
        from paper_2607_06827_amd.workload import TrainJob
        tj = TrainJob(inputs.PREFILL_1500)
        tj.run_forward()
        tj.run_backward()  # attention backward (dQ, then dK/dV), pooling backward (+ du sum)
        src = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"traffic_run": True, "train": True, "workload": tj.wl.name,
                          "copy_bytes": 1 << 30, "attn_bwd_flops": tj.attn_bwd_flops(),
                          "attn_bwd_bytes": tj.attn_bwd_bytes(), "pool_bwd_bytes": tj.pool_bwd_bytes()}))
        return
    log(f"building {wl.name} on {torch.cuda.get_device_name(0)}")
    t0 = time.perf_counter()
    job = Job(wl, num_splits=args.num_splits)
    torch.cuda.synchronize()
    log(f"inputs and caches ready in {time.perf_counter() - t0:.1f} s")
    if args.traffic:
        job.run()  # the step's launches, eagerly: 28 pool, 28 prefill, 128 x 28 decode
        from paper_2607_06827_amd.workload import HiddenPoolJob
        hj = HiddenPoolJob(wl)
        hj.run()  # one HS Compression pooling launch of the same batch
        src = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)  # 1 GiB read + 1 GiB written by one copy kernel
        torch.cuda.synchronize()
        dec_bytes, launches = decode_launch_stats(job)
        nl = len(job.layers)
        print(json.dumps({"traffic_run": True, "workload": wl.name, "copy_bytes": 1 << 30,
                          "decode_bytes_per_launch": dec_bytes / max(launches, 1), "decode_launches": launches,
                          "pool_bytes_per_launch": sum(job.pool_bytes_layer(i) for i in range(nl)) / nl,
                          "prefill_flops_per_launch": sum(job.prefill_flops_layer(i) for i in range(nl)) / nl,
                          "hs_pool_bytes_per_launch": hj.bytes(), "layers": nl}))
        return
    pooled = measure(job, args.steps, args.warmup, "pooled (l0=14, w=4)")

    full = None
    if not args.no_full:
        fjob = Job(wl, l0=wl.num_layers, share_inputs=job, num_splits=args.num_splits)
        full = measure(fjob, args.steps, args.warmup, "full KV")
        del fjob
        torch.cuda.empty_cache()

    extras = {}
    if not args.no_extras:
        extras["fused_prefill"] = measure_fused(job, args.steps)
        torch.cuda.empty_cache()
        extras["multi_turn"] = measure_segments(args.steps)
        torch.cuda.empty_cache()
        adaptive = measure_adaptive(job, args.steps, args.warmup, args.num_splits)
        adaptive["speedup_over_uniform_w"] = adaptive["tokens_per_s"] / pooled["tokens_per_s"]
        extras["adaptive_w"] = adaptive
        torch.cuda.empty_cache()
        extras["hs_pool"] = measure_hs_pool(wl, args.steps)
        torch.cuda.empty_cache()
        extras["train_bwd"] = measure_train_bwd(args.steps)
        torch.cuda.empty_cache()
        extras["prefill_1596"] = measure_prefill_1596(args.steps)
        torch.cuda.empty_cache()
        extras["long_10min"] = measure_long_sweep(args.steps)
        torch.cuda.empty_cache()

    dec_bytes, launches = decode_launch_stats(job)
    avg_launch_ms = pooled["decode_ms"] / launches
    achieved = dec_bytes / launches / (avg_launch_ms * 1e-3) / 1e9
    log("measuring the attainable streaming-read rate")
    ceiling = stream_ceiling(job)
    cls = pooled["decode_classes"]
    result = {
        "metric": METRIC,
        "value": pooled["tokens_per_s"],
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": pooled["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": wl.name, "batch": wl.batch, "layers": wl.num_layers,
                   "l0": wl.l0, "w": wl.w, "prefix_tokens": wl.prefix_len,
                   "speech_frames": wl.speech_len, "decode_steps": wl.decode_steps,
                   "q_heads": wl.num_q_heads, "kv_heads": wl.num_kv_heads,
                   "head_dim": wl.head_dim, "page_size": wl.page_size,
                   "tokens_per_step": wl.batch * wl.decode_steps},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBPS, "traffic": measured_traffic(),
                     "kernel": "decode_kernel (+ split merge)",
                     "avg_launch_us": avg_launch_ms * 1e3,
                     "bytes_per_launch": dec_bytes / launches,
                     "attainable": dict(ceiling, frac=achieved / ceiling["gbps"]),
                     "pooled_frac": cls.get("pooled", {}).get("achieved_gbps", 0) / HBM_PEAK_GBPS,
                     "full_frac": cls.get("full", {}).get("achieved_gbps", 0) / HBM_PEAK_GBPS,
                     "pooled_frac_of_attainable": (cls.get("pooled", {}).get("achieved_gbps", 0)
                                                   / ceiling["pooled_launch_gbps"]
                                                   if ceiling.get("pooled_launch_gbps") else None),
                     "full_frac_of_attainable": (cls.get("full", {}).get("achieved_gbps", 0)
                                                 / ceiling["full_launch_gbps"]
                                                 if ceiling.get("full_launch_gbps") else None),
                     "classes": cls},
        "decode": {"pooled_tokens_per_s": pooled["decode_tokens_per_s"],
                   "pooled_gbps": pooled["decode_gbps"], "pooled_ms_per_step": pooled["decode_ms"]},
        "prefill_ms": pooled["prefill_ms"],
        "pool": pooled["pool"],
        "prefill_attn": pooled["prefill_attn"],
        **extras,
    }
    if full:
        result["full_kv"] = {"tokens_per_s": full["tokens_per_s"], "ms_per_step": full["ms_per_step"],
                             "decode_tokens_per_s": full["decode_tokens_per_s"],
                             "decode_gbps": full["decode_gbps"], "prefill_ms": full["prefill_ms"],
                             "speedup_pooled_over_full": pooled["tokens_per_s"] / full["tokens_per_s"],
                             "decode_speedup": pooled["decode_tokens_per_s"] / full["decode_tokens_per_s"]}
    if not args.no_cpu:
        log("timing the CPU oracle on a sample of the job")
        result["cpu_baseline"] = cpu_baseline(job)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
