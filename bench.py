#!/usr/bin/env python3
"""Benchmark of the OmniCache cached attention layer on one MI355X.

Workload: an SD3-1024-like joint-attention layer (64x64 = 4096 image tokens
plus 333 uncached text tokens, C=1536, 24 heads x 64, bf16) with Token Cache
at ratio r, seeded synthetic inputs (oc_synth), weights ~ N(0, 1/C).  One
"step" is one oc_layer_cached call on a new denoising-step input with a warm
layer cache: match, select, reduced attention, in-place restoration.

Prints one JSON line: throughput in layer tokens per second at r (default
0.5), latency and speed-up against the uncached layer at r = 0.25/0.5/0.75,
the roofline of the dominant kernel (live HIP-event stage timing), and the
CPU oracle timed on a bounded sample on this host.
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "cached attn-layer tokens/sec & latency vs uncached at r; MFMA % / HBM GB/s"
PEAK_MFMA_TFLOPS = 2516.6     # MI355X dense bf16 / fp16 MFMA
PEAK_HBM_GBS = 8000.0         # MI355X HBM3E
# Counter summary of the dominant kernel (rocprofv3 FETCH_SIZE / WRITE_SIZE
# runs, scaled by a copy kernel of known size) and the sources it was taken on.
PROFILE = os.path.join(ROOT, "profiles", "sd3_1024_r050_kernels.md")
FLASH_SOURCES = ("k_flash.hip", "oc_attn_common.h", "oc_device.h")


def flash_source_hash():
    import hashlib
    h = hashlib.sha1()
    for f in FLASH_SOURCES:
        with open(os.path.join(ROOT, "paper_2607_23844_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def flash_traffic():
    """HBM bytes per flash launch from the committed counter summary, or None
    when there is none or the kernel's sources changed since it was taken."""
    try:
        with open(PROFILE) as fh:
            kv = dict(l.split(":", 1) for l in fh.read().splitlines() if l.startswith("flash_"))
        if kv["flash_source_sha1"].strip() != flash_source_hash():
            return None
        return int(float(kv["flash_traffic_bytes_per_launch"]))
    except (OSError, KeyError, ValueError):
        return None


def stage_work(shape, pl, n_ctx):
    """Algorithmic work per launch of each stage: (kind, amount, unit)."""
    C, H, dh = shape.C, shape.heads, shape.head_dim
    hd = H * dh
    rows = pl.n_kept + n_ctx
    FN = shape.F * shape.N
    lk = pl.seq_len + (n_ctx if pl.n_seq == 1 else 0)
    attn_flop = 4.0 * pl.n_seq * lk * lk * hd
    S, D, G = pl.n_src_max, pl.n_dst_max, pl.n_groups
    return {
        "proj_qk": ("mfma", 2.0 * rows * C * 2 * hd),
        "proj_v": ("mfma", 2.0 * rows * C * hd),
        "flash": ("mfma", attn_flop),
        "proj_out": ("mfma", 2.0 * rows * hd * C),
        "match": ("mfma", 2.0 * G * S * D * C),
        "inv_norm": ("hbm", FN * C * 2.0 + FN * 4.0),
        "gather": ("hbm", 2.0 * pl.n_kept * C * 2.0),
        "restore": ("hbm", 2.0 * pl.n_kept * C * 2.0),
    }


def run_gpu(args):
    import numpy as np
    import torch
    import paper_2607_23844_amd as oc
    from paper_2607_23844_amd.runner import FullRunner, LayerRunner
    from oc_synth import make_workload

    dev = torch.device("cuda:0")
    wl = make_workload("sd3_1024", 4)
    shape = oc.Shape(wl.F, wl.H, wl.W, wl.C, wl.heads, wl.head_dim, wl.n_ctx, "bf16")

    def t(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev)

    xs = [t(s) for s in wl.steps]
    ctx = t(wl.ctx)
    W = {k: t(getattr(wl, k)) for k in ("wq", "wk", "wv", "wo")}
    tokens = shape.F * shape.N + shape.n_ctx
    K, Wm = args.steps, args.warmup

    def timed(fn, inputs):
        for i in range(Wm):
            fn(inputs[i % len(inputs)])
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0 = time.perf_counter()
        e0.record()
        for i in range(K):
            fn(inputs[i % len(inputs)])
        e1.record()
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        return e0.elapsed_time(e1) / K, wall

    full = FullRunner(shape, oc.Cfg("token", 0.0), W, dev, ctx)
    full_ms, _ = timed(full, xs)
    by_r = {}
    primary = None
    for r in sorted(set([0.25, 0.5, 0.75, args.r])):
        cfg = oc.Cfg("token", r=r, patch_k=1)
        run = LayerRunner(shape, cfg, W, dev, ctx)
        run(xs[0])                       # cold step: the layer cache becomes valid
        ms, wall = timed(run, xs[1:])
        by_r[str(r)] = dict(ms=ms, tokens_per_s=tokens / (ms * 1e-3), speedup_vs_uncached=full_ms / ms)
        if r == args.r:
            primary = (cfg, run, ms, wall)
    cfg, run, ms, wall = primary
    # live per-kernel timing: HIP events stamped by the runtime at each kernel's start and end
    timer = oc.StageTimer()
    with timer:
        for i in range(K):
            run(xs[1 + i % 3])
    torch.cuda.synchronize()
    stages = timer.collect()
    pl = oc.plan(shape, cfg)
    work = stage_work(shape, pl, shape.n_ctx)
    kernels = {}
    for name, (tot_ms, n) in stages.items():
        avg_us = tot_ms * 1e3 / max(n, 1)
        d = dict(avg_us=round(avg_us, 3), launches_per_step=n / K)
        if name in work:
            kind, amount = work[name]
            if kind == "mfma":
                ach = amount / (avg_us * 1e-6) / 1e12
                d.update(bound="mfma", achieved_tflops=round(ach, 2), frac=round(ach / PEAK_MFMA_TFLOPS, 4))
            else:
                ach = amount / (avg_us * 1e-6) / 1e9
                d.update(bound="hbm", achieved_gbs=round(ach, 1), frac=round(ach / PEAK_HBM_GBS, 4))
        kernels[name] = d
    dom = max(stages, key=lambda s: stages[s][0])
    dom_avg_us = stages[dom][0] * 1e3 / stages[dom][1]
    roof = None
    traffic = flash_traffic() if dom == "flash" else None
    if dom in work:
        kind, amount = work[dom]
        if kind == "mfma":
            ach = amount / (dom_avg_us * 1e-6) / 1e12
            roof = dict(kernel=dom, bound="mfma", achieved=round(ach, 2), peak=PEAK_MFMA_TFLOPS, unit="TFLOP/s",
                        frac=round(ach / PEAK_MFMA_TFLOPS, 4), traffic=traffic, avg_us=round(dom_avg_us, 3),
                        algorithmic_per_launch=amount)
        else:
            ach = amount / (dom_avg_us * 1e-6) / 1e9
            roof = dict(kernel=dom, bound="hbm", achieved=round(ach, 1), peak=PEAK_HBM_GBS, unit="GB/s",
                        frac=round(ach / PEAK_HBM_GBS, 4), traffic=traffic, avg_us=round(dom_avg_us, 3),
                        algorithmic_per_launch=amount)
    return dict(ms=ms, wall=wall, tokens=tokens, full_ms=full_ms, by_r=by_r, kernels=kernels, roofline=roof,
                plan=dict(n_kept=pl.n_kept, n_cached=pl.n_cached, seq_len=pl.seq_len))


def run_cpu_baseline(args):
    """The CPU oracle, unchanged, single-threaded, on a bounded sample: a cold
    step then warm steps of the same layer."""
    from threadpoolctl import threadpool_limits
    from oc_synth import make_workload
    from oracle import oc_oracle as O

    wl = make_workload("sd3_1024", 1 + args.cpu_steps)
    sh = O.LayerShape(wl.F, wl.H, wl.W, wl.C, wl.heads, wl.head_dim, wl.n_ctx)
    cf = O.CacheCfg("token", r=args.r)
    W = {k: wl.f64(getattr(wl, k)) for k in ("wq", "wk", "wv", "wo")}
    ctx = wl.f64(wl.ctx)
    with threadpool_limits(1):
        r0 = O.layer_step(wl.f64(wl.steps[0]), ctx, W, sh, cf, None, False)
        t0 = time.perf_counter()
        cache = r0.y
        for s in range(1, 1 + args.cpu_steps):
            cache = O.layer_step(wl.f64(wl.steps[s]), ctx, W, sh, cf, cache, True).y
        dt = (time.perf_counter() - t0) / args.cpu_steps
    tokens = wl.F * wl.N + wl.n_ctx
    return dict(value=round(tokens / dt, 2), unit="tokens/s", cores=1, kind="oracle",
                sample=f"{args.cpu_steps} warm steps of the full layer (4096+333 tokens, r={args.r}), fp64 NumPy, "
                       f"one thread; {dt:.2f} s per step; host has {os.cpu_count()} logical CPUs "
                       f"({platform.processor() or platform.machine()})")


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--r", type=float, default=0.5)
    ap.add_argument("--cpu-steps", type=int, default=2)
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--copy-probe", action="store_true",
                    help="first run a plain 256 MiB read + 256 MiB write elementwise kernel (counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on exactly one GPU: the cached layer is measured whole on a single MI355X and there is "
              f"no multi-GPU path (asked for --gpus {args.gpus})", file=sys.stderr)
        sys.exit(2)
    if args.copy_probe:
        import torch
        src = torch.ones(64 << 20, dtype=torch.float32, device="cuda:0")
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.mul(src, 1.0, out=dst)
        torch.cuda.synchronize()
        del src, dst
    g = run_gpu(args)
    cpu = None if args.no_cpu else run_cpu_baseline(args)
    ms = g["ms"]
    line = {
        "metric": METRIC,
        "value": round(g["tokens"] / (ms * 1e-3), 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": f"SD3-1024-like joint-attention layer, Token Cache r={args.r}: F=1, 64x64 image tokens + "
                        f"333 uncached text tokens, C=1536, 24 heads x 64, bf16, patch_k=1, warm layer cache",
            "r": args.r,
            "tokens_per_step": g["tokens"],
            "retained_image_tokens": g["plan"]["n_kept"],
        },
        "latency_us": round(ms * 1e3, 2),
        "uncached_latency_us": round(g["full_ms"] * 1e3, 2),
        "speedup_vs_uncached": round(g["full_ms"] / ms, 4),
        "by_r": {k: {kk: round(vv, 4) for kk, vv in v.items()} for k, v in g["by_r"].items()},
        "roofline": g["roofline"],
        "kernels": g["kernels"],
        "cpu_baseline": cpu,
        "wall_s_timed_region": round(g["wall"], 4),
    }
    print(json.dumps(line))


if __name__ == "__main__":
    main()
