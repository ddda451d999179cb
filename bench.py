"""Benchmark: SMA training throughput of k learners on one MI355X.

One step = one SMA iteration of the whole hot path: every learner's forward
and backward pass on its batch (cb_step) and the fused synchronisation
(cb_sync).  The headline workload is ResNet-32 replicas (CIFAR-shaped
synthetic images), k = 4 learners of batch 32.  Also reported in the same
JSON line: a sweep over k at batch 16, the SMA-only microbenchmark (ResNet-50's
25.6M parameters x 32 replicas, HBM GB/s), and the oracle timed on the host.

python bench.py [--gpus 1] [--steps K] [--warmup W]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0        # MI355X HBM3E
FP32_MFMA_PEAK_TFS = 157.3   # MI355X dense fp32 matrix


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def _ring(wk, n, dev):
    import torch
    import workloads as wl

    xs, ys = [], []
    for t in range(n):
        x, y = wl.batch(wk.n_images, wk.in_c, wk.in_h, wk.in_w, wk.num_classes, wk.seed, t)
        xs.append(torch.from_numpy(x).to(dev))
        ys.append(torch.from_numpy(y).to(dev))
    return xs, ys


def roofline_of(prof):
    """Roofline object for the kernel with the largest total time in a
    profile {name: (launches, ms, flops, bytes)}."""
    name, (la, ms, fl, by) = max(prof.items(), key=lambda kv: kv[1][1])
    if fl > 0:
        ach = fl / (ms * 1e-3) / 1e12
        return {"kernel": name, "bound": "mfma", "achieved": round(ach, 3),
                "peak": FP32_MFMA_PEAK_TFS, "unit": "TFLOP/s",
                "frac": round(ach / FP32_MFMA_PEAK_TFS, 4), "traffic": None,
                "launches": la, "avg_launch_us": round(ms * 1e3 / la, 2),
                "algorithmic_per_launch": fl / la}
    ach = by / (ms * 1e-3) / 1e9
    return {"kernel": name, "bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS,
            "unit": "GB/s", "frac": round(ach / HBM_PEAK_GBS, 4), "traffic": None,
            "launches": la, "avg_launch_us": round(ms * 1e3 / la, 2),
            "algorithmic_per_launch": by / la}


def time_training(wk, steps, warmup, ring=8, prof_steps=0):
    """ms per SMA iteration (cb_step + cb_sync) for workload wk."""
    import torch
    import paper_1901_02244_amd as cb
    import workloads as wl

    m = cb.model(wk.arch, wk.in_c, wk.in_h, wk.in_w, wk.num_classes)
    w0 = wl.init_w0(cb.cb_tensor_layout(m), wk.seed)
    ctx = cb.Context(m, wk.k, wk.b, wk.alpha, wk.lr, wk.momentum, w0)
    xs, ys = _ring(wk, min(ring, steps + warmup), "cuda")
    n = len(xs)
    for i in range(warmup):
        ctx.cb_step(xs[i % n], ys[i % n])
        ctx.cb_sync()
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    ev0.record()
    for i in range(steps):
        ctx.cb_step(xs[i % n], ys[i % n])
        ctx.cb_sync()
    ev1.record()
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) * 1e3 / steps
    ms = ev0.elapsed_time(ev1) / steps
    loss = ctx.cb_get_loss()
    prof = None
    if prof_steps:
        # per-kernel durations: every launch carries start/stop events on its
        # own dispatch (hipExtLaunchKernel), on the context's stream; the same
        # loop as the timed one, run again with instrumentation on
        ctx.cb_profile_enable(True)
        pe0, pe1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        pe0.record()
        for i in range(prof_steps):
            ctx.cb_step(xs[i % n], ys[i % n])
            ctx.cb_sync()
        pe1.record()
        torch.cuda.synchronize()
        prof = ctx.cb_profile()
        ctx.cb_profile_enable(False)
        prof = {k: (v[0] / prof_steps, v[1] / prof_steps, v[2] / prof_steps, v[3] / prof_steps)
                for k, v in prof.items()}
        log(f"[bench] {wk.name}: instrumented pass {pe0.elapsed_time(pe1) / prof_steps:.3f} ms/step "
            f"(kernel sum {sum(v[1] for v in prof.values()):.3f} ms)")
    ctx.close()
    del ctx
    torch.cuda.empty_cache()
    if prof_steps:
        return ms, wall, loss, prof
    return ms, wall, loss


def sma_micro(steps=20, warmup=3):
    """Fused SMA kernel alone on ResNet-50's P with k = 32 replicas."""
    import torch
    import paper_1901_02244_amd as cb
    import workloads as wl

    k = wl.SMA_MICRO_K
    m = cb.model("resnet50", 3, 224, 224, 1000)
    P = cb.cb_num_params(m)
    w0 = wl.init_w0(cb.cb_tensor_layout(m), 4)
    ctx = cb.Context(m, k, 1, 1.0 / k, 0.01, 0.9, w0)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(7)
    g = torch.randn((k, P), generator=gen, device="cuda", dtype=torch.float32) * 0.05
    for _ in range(warmup):
        ctx.cb_sma_apply(g)
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record()
    for _ in range(steps):
        ctx.cb_sma_apply(g)
    ev1.record()
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / steps
    nbytes = 4 * P * (3 * k + 4)
    ctx.cb_profile_enable(True)
    for _ in range(steps):
        ctx.cb_sma_apply(g)
    prof = ctx.cb_profile()
    ctx.close()
    del ctx, g
    torch.cuda.empty_cache()
    la, kms, _, kby = prof["sma_k"]
    return {"P": P, "k": k, "ms": round(ms, 4), "bytes": nbytes,
            "GB/s": round(nbytes / ms / 1e6, 1), "frac_hbm": round(nbytes / ms / 1e6 / HBM_PEAK_GBS, 4),
            "kernel_avg_us": round(kms * 1e3 / la, 2),
            "kernel_GB/s": round(kby / (kms * 1e-3) / 1e9, 1),
            "kernel_frac_hbm": round(kby / (kms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}


def cpu_baseline(wk):
    """The oracle as it stands: one SMA iteration of the same workload on one core."""
    import oracle
    import workloads as wl

    m = oracle.model(wk.arch, wk.in_c, wk.in_h, wk.in_w, wk.num_classes)
    w0 = wl.init_w0(oracle.tensors(m), wk.seed)
    ref = oracle.SMA(m, w0, wk.k, wk.b, wk.alpha, wk.lr, wk.momentum)
    x, y = wl.workload_batch(wk, 0)
    t0 = time.perf_counter()
    ref.step(x, y)
    ref.sync()
    dt = time.perf_counter() - t0
    return {"value": round(wk.n_images / dt, 3), "unit": "images/s", "cores": 1, "kind": "oracle",
            "sample": f"1 SMA iteration of {wk.name} ({wk.n_images} images, all {wk.k} learners "
                      f"+ sync), single-threaded, {dt:.1f} s"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--sweep-steps", type=int, default=20)
    ap.add_argument("--no-sweep", action="store_true")
    ap.add_argument("--no-micro", action="store_true")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--prof-steps", type=int, default=50)
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="first run one plain copy kernel of this many MiB (read and written once "
                         "each), the reference dispatch for HBM byte counters")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: this build runs all k learners on a single MI355X "
              f"(--gpus {args.gpus} is not supported)", file=sys.stderr)
        sys.exit(2)

    import torch
    import workloads as wl

    torch.cuda.set_device(0)
    if args.calib_copy_mib:
        n = args.calib_copy_mib * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        torch.neg(src, out=dst)  # one elementwise kernel: n floats in, n floats out
        torch.cuda.synchronize()
        log(f"[bench] copy kernel: {n * 4} bytes read, {n * 4} bytes written")
        del src, dst
        torch.cuda.empty_cache()
    wk = wl.RESNET32_K4
    log(f"[bench] {wk.name}: warmup {args.warmup}, steps {args.steps}")
    ms, wall, loss, prof = time_training(wk, args.steps, args.warmup, prof_steps=args.prof_steps)
    value = wk.n_images / (ms / 1e3)
    log(f"[bench] {wk.name}: {ms:.3f} ms/step (wall {wall:.3f}), {value:.0f} images/s")
    roof = roofline_of(prof)
    tot = sum(v[1] for v in prof.values())
    kernels = {k: {"launches_per_step": v[0], "ms_per_step": round(v[1], 4),
                   "share": round(v[1] / tot, 4),
                   "TFLOP/s": round(v[2] / (v[1] * 1e-3) / 1e12, 2) if v[2] else None,
                   "GB/s": round(v[3] / (v[1] * 1e-3) / 1e9, 1)}
               for k, v in sorted(prof.items(), key=lambda kv: -kv[1][1])}
    for k_, v_ in kernels.items():
        log(f"[bench]   {k_}: {v_}")
    log(f"[bench] roofline: {roof}")

    sweep = {}
    if not args.no_sweep:
        base = wl.RESNET32_SWEEP
        for k in base.sweep_k:
            w = base.with_k(k)
            sms, swall, _ = time_training(w, args.sweep_steps, 3)
            sweep[str(k)] = {"ms_per_step": round(sms, 4), "images_per_s": round(w.n_images / (sms / 1e3), 1)}
            log(f"[bench] sweep b=16 k={k}: {sms:.3f} ms/step, {w.n_images / (sms / 1e3):.0f} images/s")
    micro = None
    if not args.no_micro:
        micro = sma_micro()
        log(f"[bench] SMA micro: {micro}")
    cpu = None
    if not args.no_cpu:
        cpu = cpu_baseline(wk)
        log(f"[bench] cpu baseline: {cpu}")

    out = {
        "metric": "training images/sec/GPU (all k replicas) vs k; fused SMA kernel HBM GB/s",
        "value": round(value, 1),
        "unit": "images/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": f"{wk.name}: ResNet-32 replicas, 32x32x3 N(0,1) images, 10 classes, "
                               f"k={wk.k} learners x b={wk.b}, alpha=1/k, lr={wk.lr}, mu={wk.momentum}, "
                               "one SMA iteration per step",
                   "k": wk.k, "b": wk.b, "images_per_step": wk.n_images},
        "roofline": roof,
        "kernels_per_step": kernels,
        "k_sweep_b16": sweep,
        "sma_microbench": micro,
        "cpu_baseline": cpu,
        "final_loss": [round(float(v), 4) for v in loss],
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
