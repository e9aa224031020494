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
    # --no-profile --no-cpu-baseline --no-full-suffix --no-mfma --no-gen-sweep`:
    # per-dispatch means of the block-start launches (grid 393216, 376 rows) and
    # the cached ones (grid 131072, 120 rows), for the one-pass layers and the
    # layers that keep the bfloat16 pair; copy kernel: 268435456 bytes read and
    # written per launch read as 131086.1 KiB fetched and 262144.0 KiB written
    ("llada_gen256", "gemm_gate_up"): {
        "sources_sha256": "e9babf06dc649fb394273589dd248cba4496b0fc516fce905c7a3482e53c1c55",
        "fetch_kib": {"start": (135810.6, 189390.7), "cached": (104448.8, 110535.8)},
        "write_kib": {"start": (9024.0, 18048.0), "cached": (2880.0, 5760.0)},
        "fetch_scale": 262144.0 / 131086.1, "write_scale": 1.0},
}
GEMM_SOURCES = ("gemm.hip", "internal.h", "common.h")


def gemm_sources_sha256():
    h = hashlib.sha256()
    for f in GEMM_SOURCES:
        with open(os.path.join(ROOT, "paper_2608_23167_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(workload, kernel, n_layers, n_pair, start_frac):
    """Bytes per launch: the counters weighted n_pair : n_layers - n_pair over
    the layers and start_frac : 1 - start_frac over block-start and cached
    steps, as in the timed schedule; None if the sources changed since."""
    t = TRAFFIC.get((workload, kernel))
    if not t or t["sources_sha256"] != gemm_sources_sha256():
        return None

    def mix(table):
        by_kind = {k: ((n_layers - n_pair) * one + n_pair * pair) / n_layers
                   for k, (one, pair) in table.items()}
        return start_frac * by_kind["start"] + (1.0 - start_frac) * by_kind["cached"]
    return round((mix(t["fetch_kib"]) * t["fetch_scale"] + mix(t["write_kib"]) * t["write_scale"])
                 * 1024)


def n_pair_layers(dm):
    """Layers whose projection inputs keep the bfloat16 pair (two MFMA passes)."""
    from paper_2608_23167_amd import _lib as L
    cm = dm.c_model
    return {L.SSM_ACT_BF16X2: cm.n_layers,
            L.SSM_ACT_BF16X2_FIRST: min(cm.pair_layers, cm.n_layers)}.get(cm.act_mode, 0)


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
    ap.add_argument("--batch", type=int, default=None, help="override the workload's batch size")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--attn-sweep", action="store_true",
                    help="instead of the decoding bench: the attention/gather microbenchmark "
                         "(LLaDA-8B heads, batch 8, prefix 4096, block 64, suffix 4096) over the "
                         "kept-suffix count")
    ap.add_argument("--gen-sweep", action="store_true",
                    help="instead of the decoding bench: whole generations of the LLaDA-8B shape "
                         "(prompt 1024, block 64, top-8, budgets 128/32/16, prefix cache) at "
                         "generation lengths 256 .. 2048, SSM and unpruned")
    ap.add_argument("--batch-sweep", action="store_true",
                    help="instead of the decoding bench: the LLaDA-8B gen-256 workload (prompt 256, "
                         "block 32, top-1, budgets 64/16/8, prefix cache) at batch 1 .. 32")
    ap.add_argument("--no-full-suffix", action="store_true",
                    help="skip the unpruned (full-suffix) decoder run of the same schedule")
    ap.add_argument("--no-profile", action="store_true",
                    help="skip the profiled replay (per-kernel times and roofline), e.g. under counter collection")
    ap.add_argument("--no-gen-sweep", action="store_true",
                    help="skip the generation-length sweep (whole generations at 256 .. 2048, SSM and "
                         "unpruned) that the default run reports")
    ap.add_argument("--no-mfma", action="store_true",
                    help="skip the MFMA report (projections and attention of the LLaDA-8B-shaped "
                         "generation of length 1024)")
    ap.add_argument("--cpu-layers", type=int, default=None,
                    help="layers of the CPU oracle sample (default: all; fewer are extrapolated)")
    ap.add_argument("--no-cpu-samples", action="store_true",
                    help="skip the further oracle samples (tiny generation, long-workload steps, "
                         "microbenchmark attention)")
    ap.add_argument("--cpu-reps", type=int, default=4,
                    help="repetitions of each layer of the CPU oracle sample")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py: this build runs on exactly one GPU; multi-GPU runs are not supported "
              "(sequences would shard data-parallel with no per-step exchange)", file=sys.stderr)
        sys.exit(2)

    if args.attn_sweep:
        attn_sweep()
        return
    if args.gen_sweep:
        gen_sweep()
        return
    if args.batch_sweep:
        batch_sweep()
        return

    import numpy as np
    import torch

    from synthetic import WORKLOADS, initial_tokens, make_weights
    from paper_2608_23167_amd.api import (PROFILE_TAGS, ssm_profile_enable, ssm_profile_query)
    from paper_2608_23167_amd.decoder import Decoder
    from paper_2608_23167_amd.model import DeviceModel

    wl = WORKLOADS[args.workload]
    if args.batch is not None:
        wl = wl.replace(batch=args.batch)
    shape = wl.model
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    print(f"[bench] workload {wl.name}: generating weights on the GPU", file=sys.stderr, flush=True)
    mw = make_weights(shape, seed=wl.seed, device=dev)
    dm = DeviceModel(shape, mw)
    dec = Decoder(wl, dm, device=dev)
    tok0 = initial_tokens(wl, device=dev)
    # fixed top-n rules know their schedule; confidence-driven rules (threshold,
    # margin) run whole generations through Decoder.generate, which reads the
    # masks left in the block after every step
    fixed = wl.steps_per_block() is not None

    def schedule_of(d):
        if fixed:
            return d.schedule()
        rec = []
        d.generate(tok0, pre_step=lambda j, first: rec.append((j, first)))
        torch.cuda.synchronize()
        return rec

    sched = schedule_of(dec)
    K = args.steps or len(sched)
    if not fixed:
        K = min(K, len(sched))
    W = args.warmup

    def run(n, events=None, d=dec, sch=None):
        """n steps of the schedule from a fresh generation, wrapping around."""
        sch = sch or sched
        if not fixed:
            # the first n steps of a generation, as generate() runs them
            i = [0]

            def pre(j, first):
                if events is not None:
                    events[i[0]][0].record()

            def post(j, first):
                if events is not None:
                    events[i[0]][1].record()
                i[0] += 1
            d.generate(tok0, max_steps=n, pre_step=pre, post_step=post)
            return
        d.reset(tok0)
        for i in range(n):
            j, first = sch[i % len(sch)]
            if i and i % len(sch) == 0:
                d.reset(tok0)
            if events is not None:
                events[i][0].record()
            d.step(j, first)
            if events is not None:
                events[i][1].record()

    def timed(d, sch=None):
        """W warm-up steps, then K timed steps: (wall s, per-step ms, step kinds)."""
        sch = sch or sched
        k = K if fixed else min(K, len(sch))
        run(W, d=d, sch=sch)
        torch.cuda.synchronize()
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(k)]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        run(k, ev, d=d, sch=sch)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        return wall, [a.elapsed_time(b) for a, b in ev], [sch[i % len(sch)][1] for i in range(k)], k

    def medians(step_ms, kinds):
        start_ms = [t for t, f in zip(step_ms, kinds) if f]
        cached_ms = [t for t, f in zip(step_ms, kinds) if not f]
        return {"block_start_median": round(statistics.median(start_ms), 4) if start_ms else None,
                "cached_median": round(statistics.median(cached_ms), 4) if cached_ms else None}

    print(f"[bench] warmup {W} steps", file=sys.stderr, flush=True)
    wall, step_ms, kinds, _ = timed(dec)
    # tokens decoded in the timed steps: n per step for top-n; a confidence
    # rule decodes a whole generation in its len(sched) steps
    tokens = K * wl.n_per_step * wl.batch if fixed else wl.gen_len * wl.batch * K / len(sched)
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
                     "mfma_tflops": round(tfl, 1),
                     "traffic": measured_traffic(wl.name, dom, shape.n_layers, n_pair_layers(dm),
                                                 sum(1 for i in range(K) if sched[i % len(sched)][1]) / K)})

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
        "step_latency_ms": medians(step_ms, kinds),
        "kernel_ms_per_step": {t: round(prof[t][1] / K, 4) for t in PROFILE_TAGS if prof[t][0]},
        "roofline": roof,
        "cpu_baseline": None,
    }
    print(f"[bench] profile: {result['kernel_ms_per_step']}", file=sys.stderr, flush=True)

    if not args.no_full_suffix:
        # the same schedule without suffix pruning: every suffix token is a
        # local row (the unpruned decoder SSM is measured against)
        wl_full = wl.replace(local_budget=wl.gen_len, middle_budget=0, tail_budget=0)
        dec_full = Decoder(wl_full, dm, device=dev)
        fsched = schedule_of(dec_full)
        fwall, fstep_ms, fkinds, fk = timed(dec_full, fsched)
        ftokens = tokens if fixed else wl.gen_len * wl.batch * fk / len(fsched)
        fvalue = ftokens / fwall
        del dec_full
        print(f"[bench] full suffix: {K} steps in {fwall:.3f} s -> {fvalue:.1f} tokens/s",
              file=sys.stderr, flush=True)
        result["full_suffix"] = {"value": round(fvalue, 2), "unit": "tokens/s",
                                 "steps": fk, "ms_per_step": round(fwall / fk * 1e3, 4),
                                 "step_latency_ms": medians(fstep_ms, fkinds),
                                 "ssm_speedup": round(value / fvalue, 3)}

    if not args.no_mfma and shape.dtype == "bf16" and shape == WORKLOADS["llada_long1024"].model:
        result["mfma"] = mfma_report(dm, dev)
        print(f"[bench] mfma: {result['mfma']}", file=sys.stderr, flush=True)

    if not args.no_gen_sweep and shape == WORKLOADS["llada_long2048"].model:
        result["gen_sweep"] = {
            "workload": "LLaDA-8B shape, prompt 1024, block 64, top-8, budgets 128/32/16, prefix "
                        "cache; whole generations, SSM and unpruned",
            "points": gen_sweep(dm, dev, emit=False)}

    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(wl, mw, dec, args.cpu_layers or wl.model.n_layers,
                                              args.cpu_reps)
        if shape == WORKLOADS["llada_long2048"].model and not args.no_cpu_samples:
            result["cpu_baseline"]["samples"] = cpu_samples(mw)
    print(json.dumps(result), flush=True)


PROJ_TAGS = ("gemm_qkv", "gemm_o", "gemm_gate_up", "gemm_down")


def mfma_report(dm, dev, reps=3):
    """MFMA throughput of the projections and of attention on the LLaDA-8B-shaped
    generation of length 1024 (prompt 1024, block 64, budgets 128/32/16, prefix
    cache): a block-start step of the middle block (every row, prefix included)
    and a cached step of the same block.  Times are the library's per-launch
    HIP events summed over each operation (split-K reductions and merges
    included); flops are algorithmic (2 per multiply-add, attention 4 M N_kv H
    d_h).  `issued` counts the MFMA instructions actually run: the projections
    of a layer that keeps the bfloat16 pair take two passes (hi and lo parts of
    the activations), the others one."""
    import torch
    from synthetic import WORKLOADS, initial_tokens
    from paper_2608_23167_amd import _lib as L
    from paper_2608_23167_amd.api import ssm_profile_enable, ssm_profile_query, ssm_select_count
    from paper_2608_23167_amd.decoder import Decoder

    wl = WORKLOADS["llada_long1024"]
    sh = wl.model
    d_, H, Hkv, dh, F = sh.d_model, sh.n_heads, sh.n_kv_heads, sh.head_dim, sh.ffn_dim
    # MFMA passes per projection, averaged over the layers: two where a layer
    # keeps the bfloat16 pair (hi and lo parts), one where it rounds once
    passes = 1.0 + n_pair_layers(dm) / sh.n_layers
    dec = Decoder(wl, dm, device=dev)
    tok = initial_tokens(wl, device=dev)
    j = wl.n_blocks // 2
    out = {"workload": wl.name, "block": j, "peak_tflops": BF16_PEAK_TFLOPS}
    for kind, first in (("block_start", True), ("cached", False)):
        dec.reset(tok)
        dec.step(j, True, unmask=False)          # fills the prefix cache; warm-up
        dec.step(j, first, unmask=False)
        torch.cuda.synchronize()
        ssm_profile_enable(True)
        for _ in range(reps):
            dec.step(j, first, unmask=False)
        torch.cuda.synchronize()
        ms = {t: ssm_profile_query(t)[1] / reps for t in PROJ_TAGS + ("attention",)}
        ssm_profile_enable(False)
        n_rows, _, _ = ssm_select_count(dec.params(j, first))
        M = wl.batch * n_rows
        n_keys = n_rows + (0 if first else wl.prompt_len + j * wl.block_size)
        proj_fl = sh.n_layers * 2.0 * M * d_ * ((H + 2 * Hkv) * dh + d_ + 2 * F + F)
        attn_fl = sh.n_layers * 4.0 * M * n_keys * H * dh
        proj_ms = sum(ms[t] for t in PROJ_TAGS)
        proj_tf = proj_fl / (proj_ms * 1e-3) / 1e12
        attn_tf = attn_fl / (ms["attention"] * 1e-3) / 1e12
        out[kind] = {"rows": M, "keys": n_keys,
                     "proj_ms": round(proj_ms, 3),
                     "proj_ms_by_kind": {t[5:]: round(ms[t], 3) for t in PROJ_TAGS},
                     "proj_tflops": round(proj_tf, 1),
                     "proj_frac": round(proj_tf / BF16_PEAK_TFLOPS, 4),
                     "proj_issued_frac": round(passes * proj_tf / BF16_PEAK_TFLOPS, 4),
                     "attn_ms": round(ms["attention"], 3), "attn_tflops": round(attn_tf, 1),
                     "attn_frac": round(attn_tf / BF16_PEAK_TFLOPS, 4)}
    del dec
    return out


def gen_sweep(dm=None, dev=None, emit=True):
    """Tokens/s and step latency of whole generations vs generation length, SSM
    and the unpruned decoder (every suffix token kept), on one set of LLaDA-8B
    weights: prompt 1024, block 64, top-8 per step, budgets 128/32/16, prefix
    cache, batch 1.  One warm-up generation per point.  Standalone it prints
    one JSON line; inside the default bench its points are returned."""
    import torch
    from synthetic import WORKLOADS, initial_tokens, make_weights
    from paper_2608_23167_amd.decoder import Decoder
    from paper_2608_23167_amd.model import DeviceModel
    base = WORKLOADS["llada_long2048"]
    if dm is None:
        dev = torch.device("cuda:0")
        torch.cuda.set_device(dev)
        mw = make_weights(base.model, seed=base.seed, device=dev)
        dm = DeviceModel(base.model, mw)
    points = []
    for G in (256, 512, 1024, 2048):
        wl = base.replace(gen_len=G)
        pt = {"gen_len": G}
        for name, w in (("ssm", wl), ("full", wl.replace(local_budget=G, middle_budget=0,
                                                         tail_budget=0))):
            dec = Decoder(w, dm, device=dev)
            tok0 = initial_tokens(w, device=dev)
            sched = dec.schedule()

            def gen():
                dec.reset(tok0)
                for j, first in sched:
                    dec.step(j, first)
            gen()
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            gen()
            torch.cuda.synchronize()
            wall = time.perf_counter() - t0
            pt[name] = {"seconds": round(wall, 4), "tokens_per_s": round(G / wall, 1),
                        "steps": len(sched), "ms_per_step": round(wall / len(sched) * 1e3, 3)}
            del dec
            torch.cuda.empty_cache()
        pt["ssm_speedup"] = round(pt["full"]["seconds"] / pt["ssm"]["seconds"], 3)
        print(f"[bench] gen sweep {pt}", file=sys.stderr, flush=True)
        points.append(pt)
    if not emit:
        return points
    print(json.dumps({"metric": "whole-generation tokens/s vs generation length, SSM and unpruned "
                                "(LLaDA-8B shape, prompt 1024, block 64, top-8, budgets 128/32/16)",
                      "unit": "tokens/s", "n_gpus": 1, "dtype": "bf16",
                      "data": "synthetic (seeded random-init weights, uniform random prompt ids)",
                      "points": points}), flush=True)


def batch_sweep(steps=64, warmup=4):
    """Tokens/s and step latency of the bench workload (LLaDA-8B shape, prompt
    256, gen 256, block 32, top-1, budgets 64/16/8, prefix cache) at batch 1 ..
    32: every sequence shares the schedule, so a step runs B times the rows
    over one pass of the weights.  The first `steps` steps of a generation
    (blocks 0 and 1) after `warmup`; one JSON line."""
    import torch
    from synthetic import WORKLOADS, initial_tokens, make_weights
    from paper_2608_23167_amd.api import ssm_select_count
    from paper_2608_23167_amd.decoder import Decoder
    from paper_2608_23167_amd.model import DeviceModel
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    base = WORKLOADS["llada_gen256"]
    mw = make_weights(base.model, seed=base.seed, device=dev)
    dm = DeviceModel(base.model, mw)
    points = []
    for B in (1, 2, 4, 8, 16, 32):
        wl = base.replace(batch=B)
        dec = Decoder(wl, dm, device=dev)
        tok0 = initial_tokens(wl, device=dev)
        sched = dec.schedule()
        dec.reset(tok0)
        for i in range(warmup):
            dec.step(*sched[i])
        torch.cuda.synchronize()
        dec.reset(tok0)
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(steps)]
        t0 = time.perf_counter()
        for i in range(steps):
            ev[i][0].record()
            dec.step(*sched[i])
            ev[i][1].record()
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        ms = [a.elapsed_time(b) for a, b in ev]
        cached = sorted(m for m, (_, first) in zip(ms, sched[:steps]) if not first)
        pt = {"batch": B, "tokens_per_s": round(steps * wl.n_per_step * B / wall, 1),
              "ms_per_step": round(wall / steps * 1e3, 3),
              "cached_step_ms": round(cached[len(cached) // 2], 3),
              "cached_rows": B * ssm_select_count(dec.params(1, False))[0]}
        print(f"[bench] batch sweep {pt}", file=sys.stderr, flush=True)
        points.append(pt)
        del dec
        torch.cuda.empty_cache()
    print(json.dumps({"metric": "denoised tokens/s vs batch (LLaDA-8B shape, gen 256, block 32, top-1, "
                                "budgets 64/16/8, prefix cache; steps of blocks 0-1)",
                      "unit": "tokens/s", "n_gpus": 1, "dtype": "bf16",
                      "data": "synthetic (seeded random-init weights, uniform random prompt ids)",
                      "points": points}), flush=True)


def attn_sweep(reps=10):
    """Attention over prefix KV 4096 + block 64 + kept suffix rows, and the gather
    of the kept rows of a [8, 4096, 4096] bf16 suffix tensor, for kept-suffix
    counts 0 .. 4096 (local only below 48; else local kept-48, middle 32, tail
    16; 4096 = the whole suffix).  Q, K, V ~ N(0, 1); one JSON line."""
    import torch
    from synthetic.generate import seeded_normal
    from paper_2608_23167_amd.api import (select_params, ssm_attention,
                                          ssm_attention_workspace_size, ssm_gather_rows,
                                          ssm_select_suffix)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    B, H, DH, PRE, BLK, SUF = 8, 32, 128, 4096, 64, 4096
    cap = PRE + BLK + SUF
    q_all = seeded_normal((B, H, BLK + SUF, DH), 0, "sweep.q", device=dev, dtype=torch.bfloat16)
    kc = seeded_normal((B, H, cap, DH), 0, "sweep.k", device=dev, dtype=torch.bfloat16)
    vc = seeded_normal((B, H, cap, DH), 0, "sweep.v", device=dev, dtype=torch.bfloat16)
    src = seeded_normal((B, SUF, H * DH), 0, "sweep.x", device=dev, dtype=torch.bfloat16)
    tokens = torch.zeros((1, PRE + BLK + SUF), device=dev, dtype=torch.int32)
    points = []
    for kept in (0, 16, 48, 176, 256, 512, 1024, 2048, 4096):
        lb, mb, tb = (kept, 0, 0) if kept < 48 or kept == SUF else (kept - 48, 32, 16)
        prm = select_params(PRE, BLK + SUF, BLK, 0, lb, mb, 0, tb, False)
        pos = torch.empty(BLK + SUF, device=dev, dtype=torch.int32)
        tok_c = torch.empty((1, BLK + SUF), device=dev, dtype=torch.int32)
        n_rows, n_suf, _ = ssm_select_suffix(prm, tokens, pos, tok_c, None)
        assert n_suf == kept, (kept, n_suf)
        n_q, n_keys = BLK + kept, PRE + BLK + kept
        q = q_all[:, :, :n_q].contiguous()
        out = torch.empty((B, n_q, H * DH), device=dev, dtype=torch.float32)
        ws = torch.empty(ssm_attention_workspace_size(B, H, n_q), device=dev, dtype=torch.uint8)
        spos = (pos[BLK:n_rows] - (PRE + BLK)).contiguous()
        gout = torch.empty((B, kept, H * DH), device=dev, dtype=torch.bfloat16)

        def timed(fn):
            fn()
            torch.cuda.synchronize()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            for _ in range(reps):
                fn()
            b.record()
            torch.cuda.synchronize()
            return a.elapsed_time(b) / reps * 1e3

        t_att = timed(lambda: ssm_attention(q, kc, vc, n_keys, out, ws))
        flops = 4.0 * B * H * n_q * n_keys * DH
        att_bytes = 2.0 * B * H * n_q * DH + 2 * 2.0 * B * H * n_keys * DH + 4.0 * B * n_q * H * DH
        tfl = flops / (t_att * 1e-6) / 1e12
        gbs = att_bytes / (t_att * 1e-6) / 1e9
        mfma_bound = flops / att_bytes > BF16_PEAK_TFLOPS * 1e12 / (HBM_PEAK_GBS * 1e9)
        pt = {"kept": kept, "n_q": n_q, "n_keys": n_keys, "attn_us": round(t_att, 2),
              "attn_tflops": round(tfl, 1), "attn_gbs": round(gbs, 1),
              "attn_bound": "mfma" if mfma_bound else "hbm",
              "attn_frac": round(tfl / BF16_PEAK_TFLOPS if mfma_bound else gbs / HBM_PEAK_GBS, 4)}
        if kept:
            t_g = timed(lambda: ssm_gather_rows(src, spos, gout))
            g_bytes = 2 * 2.0 * B * kept * H * DH
            pt.update({"gather_us": round(t_g, 2), "gather_gbs": round(g_bytes / (t_g * 1e-6) / 1e9, 1),
                       "gather_frac": round(g_bytes / (t_g * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)})
        print(f"[bench] sweep {pt}", file=sys.stderr, flush=True)
        points.append(pt)
    small = small_kernels_micro(dev, reps)
    print(f"[bench] sweep small kernels {small}", file=sys.stderr, flush=True)
    print(json.dumps({"metric": "attention and gather per layer vs kept-suffix count "
                                "(LLaDA-8B heads, batch 8, prefix 4096, block 64, suffix 4096)",
                      "unit": "us", "n_gpus": 1, "dtype": "bf16", "data": "synthetic N(0,1) Q/K/V",
                      "points": points, "small_kernels": small}), flush=True)


def small_kernels_micro(dev, reps=10):
    """Selection + gather of token ids (a1, a2), soft embedding (a3) and unmask +
    state scatter (a7, a8) at the microbenchmark's scale: batch 8, prefix 4096,
    block 64, suffix 4096 with budgets 128/32/16 (176 kept rows), LLaDA-8B
    embedding table (126464 x 4096 bf16), top-5 state, top-8 unmasking.  A
    block-start step (prefix rows included: 4336 rows) and a cached step (block
    and kept rows: 240) of block 0.  Times are the library's per-launch HIP
    events (kernel only, no host work).  Bytes are algorithmic: the embedding
    counts each distinct table row once."""
    import ctypes as C
    import numpy as np
    import torch
    from synthetic import WORKLOADS
    from synthetic.generate import mid_generation_state
    from paper_2608_23167_amd import _lib as L
    from paper_2608_23167_amd.api import (ssm_embed_suffix, ssm_profile_enable, ssm_profile_query,
                                          ssm_select_suffix, ssm_unmask)

    wl = WORKLOADS["attn_micro"]
    sh = wl.model
    B, d, V, k, blk = wl.batch, sh.d_model, sh.vocab, wl.topk, wl.block_size
    t_np, pi_np, pw_np, ps_np = mid_generation_state(wl, 0, 1, seed=0)
    tokens = torch.from_numpy(t_np).to(dev)
    pred_ids = torch.from_numpy(pi_np).to(dev)
    pred_w = torch.from_numpy(pw_np).to(dev)
    pred_step = torch.from_numpy(ps_np).to(dev)
    emb = (torch.randn((V, d), device=dev) * 0.02).to(torch.bfloat16)
    fake = torch.zeros(d, device=dev, dtype=torch.bfloat16)

    class _Emb:   # an embedding-table-only model description (no layers)
        c_model = L.Model(0, d, sh.n_heads, sh.n_kv_heads, sh.head_dim, sh.ffn_dim, V, sh.mask_id,
                          L.SSM_DT_BF16, float(sh.rope_base), float(sh.rms_eps), emb.data_ptr(),
                          fake.data_ptr(), emb.data_ptr(), C.cast(None, C.POINTER(L.Layer)),
                          L.SSM_ACT_BF16X2)

    def kernel_us(tag, fn):
        fn()
        torch.cuda.synchronize()
        ssm_profile_enable(True)
        for _ in range(reps):
            fn()
        torch.cuda.synchronize()
        n, ms = ssm_profile_query(tag)
        ssm_profile_enable(False)
        return ms / max(n, 1) * 1e3

    def rate(nbytes, us):
        gbs = nbytes / (us * 1e-6) / 1e9
        return {"us": round(us, 2), "bytes": int(nbytes), "gbs": round(gbs, 1),
                "frac": round(gbs / HBM_PEAK_GBS, 4)}

    out = {}
    cap = wl.total_len
    for kind, incl in (("block_start", True), ("cached", False)):
        prm = select_params_of(wl, 0, incl)
        pos = torch.empty(cap, device=dev, dtype=torch.int32)
        tok_c = torch.empty((B, cap), device=dev, dtype=torch.int32)
        region = torch.empty(cap, device=dev, dtype=torch.int8)
        n_rows, n_suf, first = ssm_select_suffix(prm, tokens, pos, tok_c, region)
        t_sel = kernel_us("select", lambda: ssm_select_suffix(prm, tokens, pos, tok_c, region))
        sel_bytes = B * n_rows * 4 * 2 + n_rows * 5          # ids gathered and written; pos, region
        x = torch.empty((B, n_rows, d), device=dev, dtype=torch.float32)
        t_emb = kernel_us("embed", lambda: ssm_embed_suffix(_Emb, tok_c, pos, region, n_rows,
                                                            pred_ids, pred_w, pred_step, 0, k,
                                                            wl.alpha, x))
        # distinct table rows the step needs, and the soft rows' state
        pos_h = pos[:n_rows].cpu().numpy()
        reg_h = region[:n_rows].cpu().numpy()
        tok_h = tok_c[:, :n_rows].cpu().numpy()
        soft = (reg_h[None, :] >= 2) & (ps_np[:, pos_h] == 0)
        rows = set(np.unique(tok_h[~soft]).tolist())
        if soft.any():
            rows |= set(np.unique(pi_np[:, pos_h][soft]).tolist()) | {sh.mask_id}
        emb_bytes = len(rows) * d * 2 + int(soft.sum()) * k * 8 + B * n_rows * d * 4
        n_out = n_rows - first
        argmax = torch.randint(0, V - 1, (B * n_out,), device=dev, dtype=torch.int32)
        conf = torch.rand(B * n_out, device=dev)
        topk_ids = torch.randint(0, V - 1, (B * n_out * k,), device=dev, dtype=torch.int32)
        topk_w = torch.rand(B * n_out * k, device=dev)
        selected = torch.zeros(B * blk, device=dev, dtype=torch.uint8)
        left = torch.zeros(B, device=dev, dtype=torch.int32)
        tok_work = tokens.clone()
        pos_out = pos[first:n_rows]
        t_unm = kernel_us("unmask", lambda: ssm_unmask(
            tok_work, wl.prompt_len, blk, sh.mask_id, L.SSM_UNMASK_TOPN, wl.n_per_step, 0.9,
            argmax, conf, topk_ids, topk_w, k, n_out, pos_out, 1, pred_ids, pred_w, pred_step,
            selected, left))
        unm_bytes = B * n_out * (8 + k * 8) + B * blk * 8 + B * n_suf * (k * 8 + 4)
        out[kind] = {"rows": n_rows, "kept": n_suf, "select": rate(sel_bytes, t_sel),
                     "embed": rate(emb_bytes, t_emb), "embed_table_rows": len(rows),
                     "unmask": rate(unm_bytes, t_unm)}
    return out


def select_params_of(wl, block_idx, include_prefix):
    from paper_2608_23167_amd.api import select_params
    return select_params(wl.prompt_len, wl.gen_len, wl.block_size, block_idx, wl.local_budget,
                         wl.middle_budget, wl.middle_mode, wl.tail_budget, include_prefix)


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
            "step_seconds": round(step_s, 3), **host_info()}


def host_info():
    """CPU model and the BLAS library NumPy runs on (threadpoolctl)."""
    model = None
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    blas = None
    try:
        from threadpoolctl import threadpool_info
        for p in threadpool_info():
            if p.get("user_api") == "blas":
                blas = f"{p.get('internal_api')} {p.get('version')} ({p.get('num_threads')} threads)"
                break
    except Exception:
        pass
    return {"cpu_model": model, "blas": blas, "nproc": os.cpu_count()}


def cpu_samples(mw_llada):
    """Further oracle samples on the host cores (bounded, about 10-30 s):
      * the tiny float32 workload: one whole generation (32 steps);
      * the long LLaDA-8B workload (prompt 1024, gen 2048, block 64, budgets
        128/32/16, prefix cache): a block-start and a cached step at the first,
        a middle and the last block, each as one decoder layer (extrapolated to
        32 layers) plus the LM head and row statistics of its output rows;
      * the attention microbenchmark (LLaDA-8B heads, batch 8, prefix 4096,
        block 64, 176 kept suffix rows): the oracle's attention of one layer.
    Inputs are synthetic rows of the step's shape; the LLaDA-shaped weights are
    those of the bench model (same shape and seed)."""
    import numpy as np
    import oracle.generate as OG
    import oracle.model as OM
    import oracle.selection as OS
    from synthetic import WORKLOADS, make_weights
    out = []
    tiny = WORKLOADS["tiny"]
    wt = OG.NumpyWeights(make_weights(tiny.model, seed=tiny.seed))
    t0 = time.perf_counter()
    _, recs = OG.generate(tiny, wt, initial_tokens_np(tiny))
    dt = time.perf_counter() - t0
    out.append({"workload": "tiny", "sample": f"whole generation ({len(recs)} steps)",
                "seconds": round(dt, 3), "tokens_per_s": round(tiny.gen_len / dt, 2)})
    print(f"[bench] cpu sample {out[-1]}", file=sys.stderr, flush=True)

    wl = WORKLOADS["llada_long2048"]
    sh = wl.model
    w = OG.NumpyWeights(mw_llada, dtype=np.float32, keep_layers=False)
    lw = w.layers[0]
    rng = np.random.default_rng(0)
    for j in (0, wl.n_blocks // 2, wl.n_blocks - 1):
        t_head = None
        for kind, incl in (("block_start", True), ("cached", False)):
            rows = OS.compacted_rows(wl.prompt_len, wl.gen_len, wl.block_size, j, wl.local_budget,
                                     wl.middle_budget, wl.middle_mode, wl.tail_budget, incl)
            n = len(rows.pos)
            x = (0.02 * rng.standard_normal((n, sh.d_model))).astype(np.float32)
            kp = vp = None
            if not incl:
                P = wl.prompt_len + j * wl.block_size
                kp = rng.standard_normal((P, sh.n_kv_heads, sh.head_dim)).astype(np.float32)
                vp = rng.standard_normal((P, sh.n_kv_heads, sh.head_dim)).astype(np.float32)
            t0 = time.perf_counter()
            y = OM.layer_forward(x, rows.pos, lw, sh, kp, vp).x
            t_layer = time.perf_counter() - t0
            if t_head is None:
                t0 = time.perf_counter()
                OM.output_stats(y[rows.first_out_row:], w, sh, wl.topk)
                t_head = time.perf_counter() - t0
            step_s = t_layer * sh.n_layers + t_head
            out.append({"workload": wl.name, "block": j, "step": kind, "rows": n,
                        "layer_seconds": round(t_layer, 3), "lm_head_seconds": round(t_head, 3),
                        "step_seconds_extrapolated": round(step_s, 2)})
            print(f"[bench] cpu sample {out[-1]}", file=sys.stderr, flush=True)

    B, H, dh, n_q, n_k = 8, 32, 128, 64 + 176, 4096 + 64 + 176
    q = rng.standard_normal((n_q, H, dh)).astype(np.float32)
    k = rng.standard_normal((n_k, H, dh)).astype(np.float32)
    v = rng.standard_normal((n_k, H, dh)).astype(np.float32)
    t0 = time.perf_counter()
    for _ in range(B):
        OM.attention(q, k, v)
    dt = time.perf_counter() - t0
    out.append({"workload": "attn_micro", "sample": f"one layer: batch {B}, {n_q} queries x {n_k} keys, "
                                                   f"{H} heads of {dh}",
                "seconds": round(dt, 3),
                "gflops": round(4.0 * B * n_q * n_k * H * dh / dt / 1e9, 1)})
    print(f"[bench] cpu sample {out[-1]}", file=sys.stderr, flush=True)
    return out


def initial_tokens_np(wl):
    from synthetic import initial_tokens
    return initial_tokens(wl).numpy()


if __name__ == "__main__":
    main()
