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
# MI355X peaks (one binary MAC counted as 2 ops):
# * popcount VALU: 256 CUs x 64 lanes x 2.4 GHz, one v_xor_b32 and one
#   v_bcnt_u32_b32 per 32 binary MACs -> 6.29e14 MAC/s = 1258 TOP/s;
# * dense MFMA: fp4 (e2m1) 10.1 PFLOP/s, int8 5.0 POP/s;
# * HBM3E 8 TB/s.
POPCOUNT_PEAK_TOPS = 256 * 64 * 2.4e9 * 32 / 2 * 2 / 1e12
FP4_PEAK_TFLOPS = 10100.0
INT8_PEAK_TOPS = 5000.0
HBM_PEAK_GBS = 8000.0
ROOT = os.path.dirname(os.path.abspath(__file__))
FWD_SOURCES = {"fwd_fp4": "paper_2412_00119_amd/csrc/k_fwd_mfma.hip",
               "fwd_popcount": "paper_2412_00119_amd/csrc/k_fwd_popcount.hip"}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def workload_macs(w, n):
    """(hidden-layer forward MACs, classifier MACs) of one step at batch n."""
    fwd = sum(n * w.widths[l] * w.widths[l - 1] for l in range(1, len(w.widths)))
    cls = sum(n * w.widths[l] * w.n_classes for l in range(1, len(w.widths)))
    return fwd, cls


def update_bytes(w):
    """Algorithmic HBM bytes of one update launch (all layers): H_l read and
    written at bits(B) bits per weight (u = (h + B) / 2 in bit planes), W_l
    written as bit rows."""
    planes = max(1, int(w.bound).bit_length())
    tot = 0
    for l in range(1, len(w.widths)):
        k_in, k_out = w.widths[l - 1], w.widths[l]
        tot += 2 * k_out * 4 * planes * ((k_in + 31) // 32) + k_out * 8 * ((k_in + 63) // 64)
    return tot


def build_sha256(rel):
    from paper_2412_00119_amd.build import kernel_fingerprint
    return kernel_fingerprint(os.path.join(ROOT, rel))


def measured_traffic(kernel, workload):
    """HBM bytes per launch of `kernel` from the committed counter summary,
    or None when there is none or the kernel source or its device compile
    flags changed since."""
    import re
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_traffic.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m_sha = re.search(r"kernel_build_sha256:\s*([0-9a-f]{64})", text)
    m_b = re.search(r"traffic_bytes_per_launch:\s*([0-9.eE+]+)", text)
    if not m_sha or not m_b or m_sha.group(1) != build_sha256(FWD_SOURCES[kernel]):
        return None
    return float(m_b.group(1))


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


def cpu_model():
    """The host CPU's model name, from /proc/cpuinfo."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or platform.machine()


def oracle_threads():
    try:
        from threadpoolctl import threadpool_info
        return max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover - threadpoolctl is optional
        return len(os.sched_getaffinity(0))


def cpu_baseline(w, budget_s=20.0, max_steps=3, first_layer_only=False):
    """The oracle, as it stands, on the first batches of the same workload:
    up to max_steps full train steps, stopping once budget_s has passed.
    With first_layer_only (a workload whose layers all have the same shape),
    each step is the oracle's step restricted to layer 1 (its forward, local
    error, selection and update: one L-th of the step's work), and the rate
    is scaled by 1/L."""
    import oracle.bmlp as ob
    from paper_2412_00119_amd import synth
    threads = oracle_threads()
    cfg = ob.Config(w.widths, w.n_classes, w.bound, w.group_size, w.robustness, w.seed_model)
    st = ob.init(cfg)
    if w.streamed:
        batches = [synth.stream_batch(w, i) for i in range(max_steps)]
    else:
        d = synth.make_split(w, "train", n=max_steps * w.batch)
        batches = list(d.batches(w.batch))
    layers = [1] if first_layer_only else None
    if first_layer_only:
        assert len(set(w.widths)) == 1, "first_layer_only needs layers of one shape"
    scale = w.n_layers if first_layer_only else 1
    steps, t0 = 0, time.perf_counter()
    for t, (x, y) in enumerate(batches):
        ob.train_step(st, x, y, t, w.p_r, layers=layers)
        steps += 1
        log(f"  oracle {w.name}: step {t} done ({time.perf_counter() - t0:.1f} s)")
        if time.perf_counter() - t0 > budget_s:
            break
    el = time.perf_counter() - t0
    fwd, cls = workload_macs(w, w.batch)
    what = (f"layer 1 of the first {steps} train step(s) (one {w.n_layers}th of each step: every layer "
            f"is {w.widths[0]}->{w.widths[1]}; rate scaled by 1/{w.n_layers})" if first_layer_only
            else f"the first {steps} full train step(s)")
    return {"value": steps * w.batch / (el * scale), "unit": "samples/s", "cores": int(threads),
            "kind": "oracle", "mac_per_s": steps * (fwd + cls) / (el * scale), "cpu_model": cpu_model(),
            "sample": f"{what} of {w.name} at batch {w.batch} from initialisation ({el:.1f} s; numpy "
                      f"float64 BLAS with {threads} threads on {cpu_model()}, "
                      f"{len(os.sched_getaffinity(0))} CPUs visible)"}


def measure(w, torch, B, steps, warmup, fwd_impl=0, max_batches=48):
    """Times one workload on the GPU.  Returns a dict with the steady-state
    step time (K steps after W warm-up steps, between two events), a
    per-kernel breakdown of the same steps (the state is put back and the
    steps run again with HIP events around each run of launches of one
    kernel class on the library's stream), and the first min(3, W) steps
    from initialisation timed one by one (every pattern is still in M_l
    there, so the update does its full Clipped-Perceptron work)."""
    net = B.BMLP(w.widths, w.n_classes, w.bound, w.batch, w.group_size, w.robustness,
                 w.seed_model, fwd_impl=fwd_impl)
    xs, ys = make_batches(w, torch, net, max_batches=max_batches)
    nb = len(xs)
    stats = torch.empty((w.n_layers, B.STATS_STRIDE), dtype=torch.int32, device="cuda")
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    t = 0

    def run(k):
        nonlocal t
        for _ in range(k):
            i = t % nb
            net.train_step(xs[i], ys[i], t, w.p_r, stats=stats)
            t += 1

    def timed(k, profile):
        torch.cuda.synchronize()
        if profile:
            B.bmlp_profile_start(net.ctx, k * (2 + 5 * w.n_layers) + 64)
        ev0.record()
        run(k)
        ev1.record()
        torch.cuda.synchronize()
        prof = B.bmlp_profile_stop(net.ctx) if profile else None
        return ev0.elapsed_time(ev1), prof

    def kernel_table(prof, k):
        return {name: {"ms_per_step": v[0] / k, "launches": v[1], "avg_launch_ms": v[0] / max(v[1], 1)}
                for name, v in prof.items()}

    # the first steps from initialisation: one by one, then again with
    # per-kernel events from the same initial state (one step first, its
    # state discarded, so that no launch below is the first of its kernel
    # in the process)
    n_first = min(3, warmup)
    init_state = net.state.clone()
    run(1)
    torch.cuda.synchronize()
    net.state.copy_(init_state)
    t = 0
    first_ms = []
    for _ in range(n_first):
        ms1, _ = timed(1, False)
        first_ms.append(ms1)
    first_counts = stats[:, :4].cpu().numpy().tolist() if n_first else None
    first = None
    if n_first:
        net.state.copy_(init_state)
        t = 0
        _, fprof = timed(n_first, True)
        first = {"steps": n_first, "ms_per_step": first_ms, "kernels": kernel_table(fprof, n_first),
                 "last_step_counts": first_counts}
    del init_state
    run(warmup - n_first)
    saved, t_saved = net.state.clone(), t
    ms, _ = timed(steps, False)
    net.state.copy_(saved)
    t = t_saved
    ms_prof, prof = timed(steps, True)
    del saved
    fwd_macs, cls_macs = workload_macs(w, w.batch)
    ms_step = ms / steps
    kernels = kernel_table(prof, steps)
    mfma = fwd_impl in (0, 2)
    fwd_avg_ms = kernels["fwd"]["avg_launch_ms"]
    macs_per_launch = fwd_macs / w.n_layers
    achieved = 2 * macs_per_launch / (fwd_avg_ms / 1e3) / 1e12
    peak = FP4_PEAK_TFLOPS if mfma else POPCOUNT_PEAK_TOPS
    upd = kernels["update"]
    upd_gbs = update_bytes(w) / (upd["avg_launch_ms"] / 1e3) / 1e9 if upd["launches"] else None
    step_tops = 2 * (fwd_macs + cls_macs) / (ms_step / 1e3) / 1e12
    out = {
        "workload": w.name, "widths": list(w.widths), "classes": w.n_classes, "bound": w.bound,
        "batch": w.batch, "steps": steps, "warmup": warmup,
        "ms_per_step": ms_step, "ms_per_step_with_kernel_events": ms_prof / steps,
        "samples_per_s": steps * w.batch / (ms / 1e3),
        "mac_per_s": (fwd_macs + cls_macs) * steps / (ms / 1e3), "mac_per_step": fwd_macs + cls_macs,
        "fwd_roofline": {"kernel": "fwd_fp4" if mfma else "fwd_popcount", "bound": "mfma" if mfma else "alu",
                         "achieved": achieved, "peak": peak, "unit": "TFLOP/s" if mfma else "TOP/s",
                         "frac": achieved / peak, "avg_launch_ms": fwd_avg_ms,
                         "launches": kernels["fwd"]["launches"],
                         "algorithmic_ops_per_launch": 2 * macs_per_launch},
        "step_roofline": {"ops_per_s_tera": step_tops,
                          "frac_popcount_alu": step_tops / POPCOUNT_PEAK_TOPS,
                          "frac_int8_mfma": step_tops / INT8_PEAK_TOPS,
                          "frac_fp4_mfma": step_tops / FP4_PEAK_TFLOPS,
                          "update_hbm_gbs": upd_gbs,
                          "update_hbm_frac": upd_gbs / HBM_PEAK_GBS if upd_gbs else None,
                          "update_bytes_per_launch": update_bytes(w)},
        "kernels": kernels,
        "first_steps": first,
    }
    return out, net, xs, ys, t


def main():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="bmlp-3072-4096x4")
    ap.add_argument("--fwd-impl", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-all-configs", action="store_true",
                    help="measure only the headline workload")
    ap.add_argument("--no-stress-oracle", action="store_true",
                    help="skip the oracle's sample of the 8192x8 workload (its state takes ~25 s to make)")
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
    log(f"workload {w.name}: widths {w.widths} c={w.n_classes} B={w.bound} bs={w.batch}")
    head, net, xs, ys, t = measure(w, torch, B, args.steps, args.warmup, fwd_impl=args.fwd_impl)
    ms_step = head["ms_per_step"]
    samples_s = head["samples_per_s"]
    kernels = head["kernels"]
    log(f"timed {args.steps} steps: {ms_step:.4f} ms/step, {samples_s:.4g} samples/s "
        f"(same steps with per-kernel events: {head['ms_per_step_with_kernel_events']:.4f} ms/step)")
    log("per-kernel ms/step: " + ", ".join(f"{k}={v['ms_per_step']:.4f}" for k, v in kernels.items()))
    if head["first_steps"]:
        log(f"first steps from initialisation: {['%.4f' % v for v in head['first_steps']['ms_per_step']]} ms")

    # Roofline of the dominant kernel, the hidden-layer forward contraction:
    # algorithmic binary MACs per launch (2 ops each) / average launch time.
    roofline = dict(head["fwd_roofline"])
    roofline["traffic"] = measured_traffic(roofline["kernel"], w.name)

    # One epoch through the epoch driver (bmlp_train_epoch: each batch
    # gathered from the device-resident training set, then stepped), over
    # the batches made above in a seeded order, timed with events on the
    # library's stream; then the error fraction and the rescaled p_r.
    epoch = None
    if not w.streamed and len(xs) > 1:
        ev0 = torch.cuda.Event(enable_timing=True)
        ev1 = torch.cuda.Event(enable_timing=True)
        x_all, y_all = torch.cat(xs), torch.cat(ys)
        order = torch.from_numpy(synth.epoch_order(w, 1, x_all.shape[0]).astype(np.int32)).cuda()
        nb = x_all.shape[0] // w.batch
        ep_stats = torch.zeros((nb, w.n_layers, B.STATS_STRIDE), dtype=torch.int32, device="cuda")
        # one batch through the driver first (untimed), so that its gather
        # kernel is not launched for the first time inside the timed region
        B.bmlp_train_epoch(net.ctx, x_all.data_ptr(), y_all.data_ptr(), x_all.shape[0], order.data_ptr(),
                           w.batch, w.batch, t, w.p_r, ep_stats.data_ptr(), net._stream())
        t += 1
        torch.cuda.synchronize()
        ev0.record()
        B.bmlp_train_epoch(net.ctx, x_all.data_ptr(), y_all.data_ptr(), x_all.shape[0], order.data_ptr(),
                           order.shape[0], w.batch, t, w.p_r, ep_stats.data_ptr(), net._stream())
        ev1.record()
        torch.cuda.synchronize()
        ep_ms = ev0.elapsed_time(ev1)
        host = ep_stats.cpu()
        err_frac, p_next = B.bmlp_epoch_summary(host.data_ptr(), nb, w.n_layers, w.batch, w.p_r)
        epoch = {"samples": nb * w.batch, "steps": nb, "ms": ep_ms,
                 "samples_per_s": nb * w.batch / (ep_ms / 1e3), "error_fraction": err_frac,
                 "p_r_next": p_next}
        log(f"one epoch through the epoch driver: {nb} steps in {ep_ms:.3f} ms "
            f"({epoch['samples_per_s']:.4g} samples/s), E = {err_frac:.4f}")
    del net, xs, ys

    # Every workload, each measured the same way (fewer steps), with the
    # oracle timed on a bounded sample of it.
    all_configs = None
    if not args.no_all_configs:
        all_configs = []
        for wc in synth.ORDERED:
            if wc.name == w.name:
                r = {k: v for k, v in head.items() if k != "kernels"}
            else:
                k_steps = 5 if wc.streamed else 20
                r, net_c, _, _, _ = measure(wc, torch, B, k_steps, 3, fwd_impl=args.fwd_impl,
                                            max_batches=6 if wc.streamed else 20)
                del net_c
                r = {k: v for k, v in r.items() if k != "kernels"}
                torch.cuda.empty_cache()
            log(f"{wc.name}: {r['ms_per_step']:.4f} ms/step, {r['samples_per_s']:.4g} samples/s, "
                f"forward at {r['fwd_roofline']['frac']:.3f} of its roof")
            all_configs.append(r)

    cpu = None
    if not args.no_cpu_baseline:
        log("timing the oracle on the host ...")
        cpu = cpu_baseline(w)
        log(f"oracle: {cpu['value']:.4g} samples/s on {cpu['cores']} threads")
        if all_configs is not None:
            for r in all_configs:
                wc = synth.WORKLOADS[r["workload"]]
                if wc.name == w.name:
                    r["oracle"] = cpu
                elif wc.streamed and args.no_stress_oracle:
                    r["oracle"] = None
                elif wc.streamed:
                    r["oracle"] = cpu_baseline(wc, budget_s=10.0, max_steps=1, first_layer_only=True)
                else:
                    r["oracle"] = cpu_baseline(wc, budget_s=10.0, max_steps=3)
                if r["oracle"]:
                    log(f"oracle {wc.name}: {r['oracle']['value']:.4g} samples/s")

    out = {
        "metric": METRIC,
        "value": samples_s,
        "unit": "samples/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "ms_per_step_with_kernel_events": head["ms_per_step_with_kernel_events"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "b1",
        "data": "synthetic",
        "config": {"workload": w.name, "widths": list(w.widths), "classes": w.n_classes,
                   "bound": w.bound, "global_batch": w.batch, "gamma": w.group_size,
                   "robustness": w.robustness, "p_r": w.p_r, "parallelism": "single-gpu"},
        "mac_per_s": head["mac_per_s"],
        "mac_per_step": head["mac_per_step"],
        "roofline": roofline,
        "step_roofline": head["step_roofline"],
        "first_steps": head["first_steps"],
        "epoch": epoch,
        "kernels": kernels,
        "cpu_baseline": cpu,
        "all_configs": all_configs,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
