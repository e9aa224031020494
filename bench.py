#!/usr/bin/env python3
"""Benchmark of SSM block-wise diffusion decoding on one MI355X.

A step is one pass of the whole hot path: suffix selection and compaction,
soft suffix embedding, the transformer forward over the compacted rows with
the prefix KV cache, LM head statistics and unmasking.  The timed region runs
K steps of the generation schedule of the workload (block-start and cached
steps in their natural mix) on a seeded random-init model; all inputs are
resident in HBM before timing starts.

Prints one JSON line: denoised tokens/s (whole job), ms per step, per-kind
step latency, the roofline of the dominant kernel (HIP events, measured in a
profiled replay of the same steps) and the CPU oracle baseline.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
FP32_PEAK_TFLOPS = 157.3

METRIC = "denoised tokens/sec + step latency per GPU (LLaDA-8B shape); % MFMA/HBM peak"

# HBM traffic of the dominant kernel per launch, from two rocprofv3 counter
# runs of this script on the same workload (FETCH_SIZE, then WRITE_SIZE, KiB
# per dispatch averaged over the kernel's dispatches), each scaled by known
# bytes / counter reading for a plain device copy.  The entry is valid only
# for the kernel sources it was measured on (sha256 of the GEMM sources).
TRAFFIC = {
    # rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE over `bench.py --steps 32 --warmup 1
    # --no-profile --no-cpu-baseline`; per-dispatch means of the block-start
    # launches (180299.2 / 18048.0 KiB) and the cached ones (106571.0 / 5760.0
    # KiB), weighted 1:31 as in the generation schedule; copy kernel:
    # 268435456 bytes read and written per launch read as 131085.1 KiB fetched
    # and 262144.0 KiB written
    ("llada_gen256", "gemm_gate_up"): {
        "sources_sha256": "d2106e91db15dfc119eec80de3d694921b7feaef98d22f5b5254d348dac21900",
        "fetch_kib": (180299.2 + 31 * 106571.0) / 32, "write_kib": (18048.0 + 31 * 5760.0) / 32,
        "fetch_scale": 262144.0 / 131085.1, "write_scale": 1.0},
}
GEMM_SOURCES = ("gemm.hip", "internal.h", "common.h")


def gemm_sources_sha256():
    h = hashlib.sha256()
    for f in GEMM_SOURCES:
        with open(os.path.join(ROOT, "paper_2608_23167_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(workload, kernel):
    t = TRAFFIC.get((workload, kernel))
    if not t or t["sources_sha256"] != gemm_sources_sha256():
        return None
    return round((t["fetch_kib"] * t["fetch_scale"] + t["write_kib"] * t["write_scale"]) * 1024)


def gemm_work(shape, tag, M):
    """Algorithmic (bytes, flops) of one projection launch over M rows."""
    es = 2 if shape.dtype == "bf16" else 4
    d, F, V = shape.d_model, shape.ffn_dim, shape.vocab
    qkv = shape.qkv_dim
    hd = shape.n_heads * shape.head_dim
    if tag == "gemm_qkv":
        N, K, out = qkv, d, M * qkv * es
    elif tag == "gemm_o":
        N, K, out = d, hd, 2 * M * d * 4          # residual read + write (fp32)
    elif tag == "gemm_gate_up":
        N, K, out = 2 * F, d, M * F * es
    elif tag == "gemm_down":
        N, K, out = d, F, 2 * M * d * 4
    elif tag == "gemm_lm_head":
        N, K, out = V, d, M * V * 4
    else:
        raise KeyError(tag)
    return N * K * es + M * K * es + out, 2.0 * M * N * K


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None, help="timed steps (default: one generation)")
    ap.add_argument("--warmup", type=int, default=8)
    ap.add_argument("--workload", default="llada_gen256")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-profile", action="store_true",
                    help="skip the profiled replay (per-kernel times and roofline), e.g. under counter collection")
    ap.add_argument("--cpu-layers", type=int, default=None,
                    help="layers of the CPU oracle sample (default: all; fewer are extrapolated)")
    ap.add_argument("--cpu-reps", type=int, default=4,
                    help="repetitions of each layer of the CPU oracle sample")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py: this build runs on exactly one GPU; multi-GPU runs are not supported "
              "(sequences would shard data-parallel with no per-step exchange)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from synthetic import WORKLOADS, initial_tokens, make_weights
    from paper_2608_23167_amd.api import (PROFILE_TAGS, ssm_profile_enable, ssm_profile_query)
    from paper_2608_23167_amd.decoder import Decoder
    from paper_2608_23167_amd.model import DeviceModel

    wl = WORKLOADS[args.workload]
    shape = wl.model
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    print(f"[bench] workload {wl.name}: generating weights on the GPU", file=sys.stderr, flush=True)
    mw = make_weights(shape, seed=wl.seed, device=dev)
    dm = DeviceModel(shape, mw)
    dec = Decoder(wl, dm, device=dev)
    tok0 = initial_tokens(wl, device=dev)
    sched = dec.schedule()
    K = args.steps or len(sched)
    W = args.warmup

    def run(n, events=None):
        """n steps of the schedule from a fresh generation, wrapping around."""
        dec.reset(tok0)
        for i in range(n):
            j, first = sched[i % len(sched)]
            if i and i % len(sched) == 0:
                dec.reset(tok0)
            if events is not None:
                events[i][0].record()
            dec.step(j, first)
            if events is not None:
                events[i][1].record()

    print(f"[bench] warmup {W} steps", file=sys.stderr, flush=True)
    run(W)
    torch.cuda.synchronize()

    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(K)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    run(K, ev)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    wall = t1 - t0
    step_ms = [a.elapsed_time(b) for a, b in ev]
    kinds = [sched[i % len(sched)][1] for i in range(K)]
    start_ms = [t for t, f in zip(step_ms, kinds) if f]
    cached_ms = [t for t, f in zip(step_ms, kinds) if not f]
    tokens = K * wl.n_per_step * wl.batch
    value = tokens / wall
    print(f"[bench] {K} steps in {wall:.3f} s -> {value:.1f} tokens/s", file=sys.stderr, flush=True)

    # profiled replay of the same steps: per-launch HIP events in the library
    prof = {t: (0, 0.0) for t in PROFILE_TAGS}
    if not args.no_profile:
        ssm_profile_enable(True)
        run(K)
        torch.cuda.synchronize()
        prof = {t: ssm_profile_query(t) for t in PROFILE_TAGS}
        main_kernel = {t: ssm_profile_query(t, 0) for t in PROFILE_TAGS}
        ssm_profile_enable(False)
    dom = max(prof, key=lambda t: prof[t][1])
    # algorithmic work of the dominant kernel over the replay
    from paper_2608_23167_amd.api import ssm_select_count
    tot_bytes = tot_flops = 0.0
    for i in range(K):
        j, first = sched[i % len(sched)]
        incl = (not wl.cache) or first
        n_rows, _, f = ssm_select_count(dec.params(j, incl))
        M = wl.batch * n_rows
        Mo = wl.batch * (n_rows - f)
        if dom.startswith("gemm_"):
            reps = 1 if dom == "gemm_lm_head" else shape.n_layers
            b_, f_ = gemm_work(shape, dom, Mo if dom == "gemm_lm_head" else M)
            tot_bytes += reps * b_
            tot_flops += reps * f_
    # the dominant operation's main kernel (split-K reductions excluded)
    n_launch, dom_ms = main_kernel[dom] if not args.no_profile else (0, 0.0)
    roof = None
    if tot_bytes > 0 and n_launch > 0:
        gbs = tot_bytes / (dom_ms * 1e-3) / 1e9
        tfl = tot_flops / (dom_ms * 1e-3) / 1e12
        intensity = tot_flops / tot_bytes
        ridge = BF16_PEAK_TFLOPS * 1e12 / (HBM_PEAK_GBS * 1e9)
        if intensity < ridge:
            roof = {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": round(gbs / HBM_PEAK_GBS, 4)}
        else:
            roof = {"bound": "mfma", "achieved": round(tfl, 1), "peak": BF16_PEAK_TFLOPS,
                    "unit": "TFLOP/s", "frac": round(tfl / BF16_PEAK_TFLOPS, 4)}
        roof.update({"kernel": dom, "launches": n_launch, "avg_launch_us": round(dom_ms / n_launch * 1e3, 2),
                     "algorithmic_bytes_per_launch": round(tot_bytes / n_launch),
                     "mfma_tflops": round(tfl, 1), "traffic": measured_traffic(wl.name, dom)})

    result = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": round(wall / K * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if shape.dtype == "bf16" else "f32",
        "data": "synthetic (seeded random-init weights N(0,0.02), uniform random prompt ids)",
        "config": {"workload": wl.name, "shape": f"{shape.n_layers}L d{shape.d_model} H{shape.n_heads}/{shape.n_kv_heads} F{shape.ffn_dim} V{shape.vocab}",
                   "batch": wl.batch, "prompt_len": wl.prompt_len, "gen_len": wl.gen_len,
                   "block": wl.block_size, "rule": f"{wl.rule}-{wl.n_per_step}",
                   "budgets": [wl.local_budget, wl.middle_budget, wl.tail_budget],
                   "prefix_cache": wl.cache, "topk": wl.topk, "alpha": wl.alpha},
        "step_latency_ms": {
            "block_start_median": round(statistics.median(start_ms), 4) if start_ms else None,
            "cached_median": round(statistics.median(cached_ms), 4) if cached_ms else None,
        },
        "kernel_ms_per_step": {t: round(prof[t][1] / K, 4) for t in PROFILE_TAGS if prof[t][0]},
        "roofline": roof,
        "cpu_baseline": None,
    }
    print(f"[bench] profile: {result['kernel_ms_per_step']}", file=sys.stderr, flush=True)

    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(wl, mw, dec, args.cpu_layers or wl.model.n_layers,
                                              args.cpu_reps)
    print(json.dumps(result), flush=True)


def cpu_baseline(wl, mw, dec, n_layers_sample, reps):
    """The oracle, untuned, on a bounded sample: one cached step at block 0 with
    `n_layers_sample` layers (each run `reps` times on the same input, the mean
    kept) plus the LM head and statistics, extrapolated to the model depth if
    fewer layers are sampled, and converted to tokens/s."""
    import numpy as np
    import oracle.generate as OG
    import oracle.model as OM
    import oracle.selection as OS
    import oracle.embed as OE
    try:
        from threadpoolctl import threadpool_info
        threads = max((p.get("num_threads", 1) for p in threadpool_info()), default=1)
    except Exception:
        threads = os.cpu_count() or 1
    print(f"[bench] cpu baseline: oracle sample ({n_layers_sample} layers) on {threads} threads",
          file=sys.stderr, flush=True)
    shape = wl.model
    w = OG.NumpyWeights(mw, dtype=np.float32, keep_layers=False)
    rows = OS.compacted_rows(wl.prompt_len, wl.gen_len, wl.block_size, 0, wl.local_budget,
                             wl.middle_budget, wl.middle_mode, wl.tail_budget, not wl.cache)
    tokens = initial_tokens_np(wl)
    pred = np.zeros((wl.total_len, wl.topk), np.int32)
    predw = np.zeros((wl.total_len, wl.topk))
    ps = np.full(wl.total_len, -1, np.int32)
    t0 = time.perf_counter()
    x = OE.embed_rows(w.tok_emb, tokens[0], rows.pos, rows.region, pred, predw, ps, -1,
                      wl.alpha, shape.mask_id)
    t_embed = time.perf_counter() - t0
    prefix = None
    if wl.cache:
        n_pre = wl.prompt_len
        rng = np.random.default_rng(0)
        prefix = [(rng.standard_normal((n_pre, shape.n_kv_heads, shape.head_dim)).astype(np.float32),
                   rng.standard_normal((n_pre, shape.n_kv_heads, shape.head_dim)).astype(np.float32))
                  for _ in range(n_layers_sample)]
    t_layers = 0.0
    for l in range(n_layers_sample):
        lw = w.layers[l]                      # conversion outside the timed part
        kp, vp = prefix[l] if prefix else (None, None)
        t0 = time.perf_counter()
        for _ in range(reps):
            y = OM.layer_forward(x, rows.pos, lw, shape, kp, vp).x
        t_layers += (time.perf_counter() - t0) / reps
        x = y
    t0 = time.perf_counter()
    OM.output_stats(x[rows.first_out_row:], w, shape, wl.topk)
    t_head = time.perf_counter() - t0
    step_s = t_embed + t_layers / n_layers_sample * shape.n_layers + t_head
    sample_s = t_embed + t_layers * reps + t_head
    return {"value": round(wl.n_per_step * wl.batch / step_s, 5), "unit": "tokens/s",
            "cores": threads, "kind": "oracle",
            "sample": (f"one cached step of {wl.name} at block 0 ({len(rows.pos)} rows): "
                       f"{n_layers_sample} of {shape.n_layers} layers (each timed {reps}x, mean) "
                       f"+ LM head and row statistics in float32 NumPy ({sample_s:.1f} s of CPU "
                       f"work) -> {step_s:.2f} s per step"),
            "step_seconds": round(step_s, 3)}


def initial_tokens_np(wl):
    from synthetic import initial_tokens
    return initial_tokens(wl).numpy()


if __name__ == "__main__":
    main()
