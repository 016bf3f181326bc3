#!/usr/bin/env python3
"""Train-step benchmark of the binary MLP library on one MI355X.

A step is one call of bmlp_train_step on one mini-batch: the bit-packed
XNOR-popcount forward of every hidden layer and of its fixed random local
classifier, the local 01-loss/robustness error signal and perceptron
selection, and the Clipped-Perceptron + reinforcement update of the int8
hidden weights with re-binarisation.  Inputs are synthetic (the Random
Prototypes recipe of the paper's Section 4.1.1 at the workload's sizes),
packed and resident in HBM before timing starts.

Prints ONE JSON line on stdout; everything else goes to stderr.

    python bench.py [--gpus 1] [--steps 50] [--warmup 5] [--workload NAME]
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

import numpy as np

METRIC = "BMLP train samples/s + XNOR-popcount MAC/s (% roofline), 4x4096 layers"
# MI355X: 256 CUs x 4 SIMD16 = 64 lanes/CU-cycle at 2.4 GHz; one v_xor_b32 and
# one v_bcnt_u32_b32 per 32 binary MACs; 1 MAC counted as 2 ops.
POPCOUNT_PEAK_TOPS = 256 * 64 * 2.4e9 * 32 / 2 * 2 / 1e12
HBM_PEAK_GBS = 8000.0


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def workload_macs(w, n):
    """(hidden-layer forward MACs, classifier MACs) of one step at batch n."""
    fwd = sum(n * w.widths[l] * w.widths[l - 1] for l in range(1, len(w.widths)))
    cls = sum(n * w.widths[l] * w.n_classes for l in range(1, len(w.widths)))
    return fwd, cls


def make_batches(w, torch, net, max_batches):
    """Packed bit rows and labels of up to max_batches batches, on the GPU."""
    from paper_2412_00119_amd import synth
    xs, ys = [], []
    if w.streamed:
        for i in range(max_batches):
            x, y = synth.stream_batch(w, i)
            xs.append(net.pack(torch.from_numpy(x).cuda()))
            ys.append(torch.from_numpy(y).cuda())
    else:
        nb = min(max_batches, w.steps_per_epoch)
        d = synth.make_split(w, "train", n=nb * w.batch)
        for x, y in d.batches(w.batch):
            xs.append(net.pack(torch.from_numpy(np.ascontiguousarray(x)).cuda()))
            ys.append(torch.from_numpy(np.ascontiguousarray(y)).cuda())
    torch.cuda.synchronize()
    return xs, ys


def cpu_baseline(w, budget_s=20.0, max_steps=3):
    """The oracle, as it stands, on the first batches of the same workload."""
    import oracle.bmlp as ob
    from paper_2412_00119_amd import synth
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover - threadpoolctl is optional
        threads = len(os.sched_getaffinity(0))
    cfg = ob.Config(w.widths, w.n_classes, w.bound, w.group_size, w.robustness, w.seed_model)
    st = ob.init(cfg)
    if w.streamed:
        batches = [synth.stream_batch(w, i) for i in range(max_steps)]
    else:
        d = synth.make_split(w, "train", n=max_steps * w.batch)
        batches = list(d.batches(w.batch))
    steps, t0 = 0, time.perf_counter()
    for t, (x, y) in enumerate(batches):
        ob.train_step(st, x, y, t, w.p_r)
        steps += 1
        if time.perf_counter() - t0 > budget_s:
            break
    el = time.perf_counter() - t0
    return {"value": steps * w.batch / el, "unit": "samples/s", "cores": int(threads),
            "kind": "oracle",
            "sample": f"{steps} full train step(s) of {w.name} at batch {w.batch} "
                      f"({el:.1f} s, numpy float64 BLAS with {threads} threads; "
                      f"host {platform.processor() or platform.machine()}, "
                      f"{len(os.sched_getaffinity(0))} CPUs visible)"}


def main():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="bmlp-3072-4096x4")
    ap.add_argument("--fwd-impl", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calib-copy-mb", type=int, default=0,
                    help="run one plain device-to-device copy of this many MiB before timing "
                         "(a known-size kernel for calibrating HBM byte counters)")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        log(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}, WORLD_SIZE {world}); "
            "the multi-GPU sharding of the step is a design note, not built.")
        sys.exit(2)

    import torch
    from paper_2412_00119_amd import synth
    from paper_2412_00119_amd import bmlp as B

    if not torch.cuda.is_available():
        log("no GPU visible")
        sys.exit(1)
    if args.calib_copy_mb > 0:
        nbytes = args.calib_copy_mb << 20
        src = torch.ones(nbytes, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"calibration copy: {nbytes} bytes read, {nbytes} bytes written")
        del src, dst
    w = synth.WORKLOADS[args.workload]
    net = B.BMLP(w.widths, w.n_classes, w.bound, w.batch, w.group_size, w.robustness,
                 w.seed_model, fwd_impl=args.fwd_impl)
    log(f"workload {w.name}: widths {w.widths} c={w.n_classes} B={w.bound} bs={w.batch}")
    xs, ys = make_batches(w, torch, net, max_batches=48)
    nb = len(xs)
    stats = torch.empty((w.n_layers, 4), dtype=torch.int32, device="cuda")
    t = 0

    def run(k):
        nonlocal t
        for _ in range(k):
            i = t % nb
            net.train_step(xs[i], ys[i], t, w.p_r, stats=stats)
            t += 1

    run(args.warmup)
    torch.cuda.synchronize()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    ev0.record()
    run(args.steps)
    ev1.record()
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1)
    ms_step = ms / args.steps
    samples_s = args.steps * w.batch / (ms / 1e3)
    fwd_macs, cls_macs = workload_macs(w, w.batch)
    log(f"timed {args.steps} steps: {ms_step:.3f} ms/step, {samples_s:.4g} samples/s")

    # Second pass over the same number of steps with every launch bracketed by
    # HIP events on the library's stream: per-kernel-class durations.
    per_step_launches = 2 + 5 * w.n_layers
    B.bmlp_profile_start(net.ctx, args.steps * per_step_launches + 64)
    run(args.steps)
    prof = B.bmlp_profile_stop(net.ctx)
    fwd_ms, fwd_n = prof["fwd"]
    fwd_avg_ms = fwd_ms / max(fwd_n, 1)
    macs_per_launch = fwd_macs / w.n_layers
    achieved = 2 * macs_per_launch / (fwd_avg_ms / 1e3) / 1e12
    kernels = {k: {"ms_per_step": v[0] / args.steps, "launches": v[1]} for k, v in prof.items()}
    log("per-kernel ms/step: " + ", ".join(f"{k}={v['ms_per_step']:.4f}" for k, v in kernels.items()))

    cpu = None
    if not args.no_cpu_baseline:
        log("timing the oracle on the host ...")
        cpu = cpu_baseline(w)
        log(f"oracle: {cpu['value']:.4g} samples/s on {cpu['cores']} threads")

    out = {
        "metric": METRIC,
        "value": samples_s,
        "unit": "samples/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "b1",
        "data": "synthetic",
        "config": {"workload": w.name, "widths": list(w.widths), "classes": w.n_classes,
                   "bound": w.bound, "global_batch": w.batch, "gamma": w.group_size,
                   "robustness": w.robustness, "p_r": w.p_r, "parallelism": "single-gpu"},
        "mac_per_s": (fwd_macs + cls_macs) * args.steps / (ms / 1e3),
        "mac_per_step": fwd_macs + cls_macs,
        "roofline": {"kernel": "fwd_popcount", "bound": "alu", "achieved": achieved,
                     "peak": POPCOUNT_PEAK_TOPS, "unit": "TOP/s", "frac": achieved / POPCOUNT_PEAK_TOPS,
                     "traffic": None, "avg_launch_ms": fwd_avg_ms, "launches": fwd_n},
        "kernels": kernels,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
