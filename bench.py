"""Benchmark of the heterogeneous data-parallel training step on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload resnet18_bf16]
                    [--no-cpu-baseline] [--no-extra] [--gpus 1]

One step = every simulated worker's forward+backward on its partition of a
synthetic CIFAR-shaped batch, the fused partition-weighted gradient average +
momentum SGD, and -- at the end of every repartition window -- the
compute-power estimate and the repartition of the next window.  By default
all workers run in one pass over the layers (hs_workers_grad: each layer is
launched once over the whole batch, with per-worker batch-norm statistics,
losses and weight gradients) and worker times follow the model clock
X_m = n_m / s_m; --streams runs one hs_worker_grad per worker on its own HIP
stream with event-measured times instead.  W untimed steps, then K timed
steps, each bracketed by HIP events on the stream the step runs on; the
batches are resident in HBM before timing.

Prints ONE JSON line:
  * value = N / median step time (samples/s); ms_per_step = the median; the
    p10 / p90 of the per-step times and the elapsed wall time;
  * step_roofline: the step's algorithmic FLOPs (fwd+bwd of every sample)
    over the median step time, against the MFMA peak of the precision;
  * kernels: every implicit-GEMM family of the step, timed with HIP events
    around its launches on the stream it runs on, in the step (two streams)
    and again with every launch on one stream (no overlap, "isolated");
  * roofline: the family with the largest time per step;
  * hbm_roofline: the fused weighted average + SGD of every timed step, and
    the same kernel alone on 8 fp32 buffers of 25M elements;
  * sim_step: the simulated synchronous step time max_m X_m;
  * the ResNet-18 fp32 (N = 1024) and VGG-16 bf16 (N = 4096) workloads'
    step time, samples/s and fractions, as sub-objects;
  * cpu_baseline: the CPU oracle's throughput on a bounded sample of the
    same step, timed on this host.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "train samples/s (fwd+bwd+wavg+SGD), CIFAR-shape ResNet-18; MFMA/HBM % peak"
ARCH_NAME = {"resnet18": "ResNet-18", "resnet50": "ResNet-50", "vgg16": "VGG-16",
             "small_cnn": "small CNN", "mlp": "MLP"}
PEAK_TFLOPS = {"bf16": 2516.6, "fp32": 157.3}   # MI355X dense MFMA peaks
HBM_PEAK_GBS = 8000.0
MODE_NAME = {0: "forward", 1: "data gradient", 2: "weight gradient"}
# every (mode, bm, bn) the step's GEMM launches can take: bm = 512 is the
# 32x32x16 MFMA 3x3 kernel with 512-row tiles, bm = bn = 64 the 64-channel
# patch kernels (modes 0 / 1) and the 3x3 weight-gradient patch kernel (mode
# 2) on the bf16 path, bm = bn = 256 the stride-2 3x3 data-gradient patch
# kernel (256 output-gradient positions x 64 channels per block, all four
# parity classes, the shortcut's data gradient summed in); the others are
# tiles of the fast implicit-GEMM kernel; (32, 64) the direct bf16 stem
# kernels (3 -> 64 channels from the fp32 NCHW batch: forward in mode 0,
# weight gradient in mode 2); (256, 128) in mode 0
# the stride-2 3x3 forward patch kernel; (64, 256) in mode 2 the stride-2
# 3x3 weight-gradient patch kernel (input as four parity planes)
PROBE_TILES = [(512, 64), (512, 128), (512, 256), (64, 64), (128, 128), (128, 64), (64, 128),
               (256, 64), (256, 256), (32, 64), (256, 128), (64, 256)]
# sub-objects of the JSON line: the other large single-GPU workloads
EXTRA = ("resnet18_fp32", "vgg16_bf16")


def kernel_name(mode, bm, bn, dtype):
    if bm == 512:
        return "conv2_kernel<%s, %dx%d tile, 32x32x16 MFMA, %s>" % (MODE_NAME[mode], bm, bn, dtype)
    if bm == 64 and bn == 256 and mode == 2:
        return "wgrad3s2_kernel<3x3 stride-2 weight gradient, 64x64x9 tile, parity planes, bf16>"
    if bm == 64 and bn == 64 and dtype == "bf16":
        if mode == 2:
            return "wgrad3_kernel<3x3 weight gradient, 64x64x9 tile, bf16>"
        return "conv64_kernel<%s, 64->64 channels 3x3 on 32x32 maps, bf16>" % MODE_NAME[mode]
    if bm == 256 and bn == 256:
        return "conv2s2_kernel<3x3 stride-2 data gradient (+1x1 shortcut), bf16>"
    if bm == 256 and bn == 128 and mode == 0:
        return "conv2s2f_kernel<3x3 stride-2 forward, 256 positions x 128 channels, bf16>"
    if bm == 32 and bn == 64:
        if mode == 2:
            return "stem_wgrad_kernel<3->64 channels 3x3 weight gradient from fp32 NCHW, bf16>"
        return "stem_fwd_kernel<3->64 channels 3x3 from fp32 NCHW, bf16>"
    return "igemm_fast_kernel<%s, %s, %dx%d tile>" % (dtype, MODE_NAME[mode], bm, bn)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="resnet18_bf16")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extra", action="store_true",
                    help="skip the other workloads' sub-objects")
    ap.add_argument("--no-probe", action="store_true",
                    help="skip the per-kernel timings")
    ap.add_argument("--cpu-samples", type=int, default=None,
                    help="samples of the CPU oracle's bounded step (default: about 15 s of "
                         "host work for the workload's network)")
    ap.add_argument("--streams", action="store_true",
                    help="one stream per worker, measured clock (default: one pass)")
    ap.add_argument("--single-stream", action="store_true",
                    help="every launch of the one-pass call on the caller's stream (per-kernel "
                         "durations without overlap, e.g. under rocprofv3)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB four times (the reference "
                         "kernel that scales the FETCH_SIZE / WRITE_SIZE counters to bytes)")
    return ap.parse_args()


# samples of the CPU oracle's bounded step per network (about 15 s of
# float64 work on the host's cores)
CPU_SAMPLES = {"resnet18": 576, "resnet50": 160, "vgg16": 2048, "small_cnn": 4096, "mlp": 65536}


def cpu_baseline(wl, seed, samples):
    """The CPU oracle (float64, numpy) on a bounded sample of the step: the same
    workers and speeds, each with its share of `samples` samples, followed by
    the weighted average and the SGD step."""
    import numpy as np
    from oracle import models as Mo
    from oracle import step as S
    from paper_2110_08941_amd import synth
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = None
    net = Mo.build(wl.arch)
    table, P = Mo.param_table(net)
    theta = synth.he_normal(table, P, seed).astype(np.float64)
    n = S.repartition(list(wl.speeds), samples) if samples >= wl.workers else [1] * wl.workers
    x, y = synth.batch(wl.in_shape, sum(n), seed, 0)
    t0 = time.perf_counter()
    out = S.step(lambda th, xm, ym: Mo.worker_grad(net, th, xm, ym), theta, None, x, y, n,
                 wl.lr, wl.mu, wl.wd)
    cp = S.estimate_cp(n, [float(v) for v in n])
    S.repartition(cp, sum(n))
    dt = time.perf_counter() - t0
    assert np.all(np.isfinite(out["theta"]))
    return {"value": round(sum(n) / dt, 3), "unit": "samples/s",
            "cores": len(os.sched_getaffinity(0)), "blas_threads": threads,
            "kind": "oracle",
            "sample": "one float64 step of %s on %d samples split %s over the %d workers "
                      "(worker gradients, weighted average, SGD, repartition); %.1f s"
                      % (wl.arch, sum(n), n, wl.workers, dt)}


def standalone_wavg(reps=20):
    """The fused weighted average + plain SGD alone on 8 fp32 gradient buffers
    of 25M elements (partition sizes of the VGG-16 workload), event-timed."""
    import torch
    from paper_2110_08941_amd import hs
    from paper_2110_08941_amd.configs import STANDALONE_WAVG as W
    P, n = W["numel"], list(W["n"])
    gen = torch.Generator(device="cuda").manual_seed(5)
    g = [torch.randn(P, device="cuda", generator=gen) for _ in n]
    th = torch.randn(P, device="cuda", generator=gen)
    ptrs = [t.data_ptr() for t in g]
    for _ in range(3):
        hs.wavg_sgd(ptrs, n, th.data_ptr(), 0, P, W["lr"], 0.0, 0.0)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        hs.wavg_sgd(ptrs, n, th.data_ptr(), 0, P, W["lr"], 0.0, 0.0)
    e1.record()
    torch.cuda.synchronize()
    us = 1e3 * e0.elapsed_time(e1) / reps
    nbytes = (len(n) * 4 + 8) * P
    del g, th
    return {"buffers": "%d x %d fp32, plain SGD" % (len(n), P), "bytes_per_launch": nbytes,
            "traffic": measured_traffic("resnet18_bf16", "wavg_sgd_kernel<2, false, false>"),
            "avg_launch_us": round(us, 2), "achieved": round(nbytes / (us * 1e-6) / 1e9, 1),
            "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(nbytes / (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)}


def attainable(reps=5):
    """What this GPU sustains on the two pipes the rooflines are priced
    against, event-timed: the MFMA loop of hs_probe_mfma_loop (dense bf16
    32x32x16 MFMAs on registers, 4 blocks of 8 waves per CU) and the plain
    1 GiB device copy of hs_probe_copy (2 GiB moved per copy)."""
    import torch
    from paper_2110_08941_amd import hs
    blocks, iters = 1024, 4000
    out = torch.empty(blocks * 512, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    hs.probe_mfma_loop(blocks, iters, out.data_ptr(), stream)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        hs.probe_mfma_loop(blocks, iters, out.data_ptr(), stream)
    e1.record()
    torch.cuda.synchronize()
    us = 1e3 * e0.elapsed_time(e1) / reps
    tf = blocks * 8 * iters * 8 * 32768 / (us * 1e-6) / 1e12
    n = (1 << 30) // 4
    src = torch.ones(n, device="cuda")
    dst = torch.empty_like(src)
    hs.probe_copy(src.data_ptr(), dst.data_ptr(), 4 * n, stream)
    e0.record()
    for _ in range(reps):
        hs.probe_copy(src.data_ptr(), dst.data_ptr(), 4 * n, stream)
    e1.record()
    torch.cuda.synchronize()
    cus = 1e3 * e0.elapsed_time(e1) / reps
    gbs = 2 * 4 * n / (cus * 1e-6) / 1e9
    del out, src, dst
    return {"mfma_bf16_loop": {"achieved": round(tf, 1), "unit": "TFLOP/s", "avg_launch_us": round(us, 1),
                               "frac_of_peak": round(tf / PEAK_TFLOPS["bf16"], 4)},
            "copy_1GiB": {"achieved": round(gbs, 1), "unit": "GB/s", "avg_launch_us": round(cus, 1),
                          "frac_of_peak": round(gbs / HBM_PEAK_GBS, 4)}}


def copy_calibration(mib, reps=4):
    """A plain device-to-device copy of a known size: under rocprofv3 --pmc its
    FETCH_SIZE and WRITE_SIZE per dispatch give the counters' scale."""
    import torch
    n = mib * (1 << 20) // 4
    src = torch.ones(n, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_per_dispatch": 4 * n, "dispatches": reps}), flush=True)


# committed HBM-traffic counter summaries, per workload
TRAFFIC_PROFILE = {"resnet18_bf16": os.path.join(ROOT, "profiles",
                                                 "hbm_traffic_resnet18_bf16_n2048_m8.md")}
# the HBM-traffic summary's entry for each probed kernel family (counted bytes per launch)
PROBE_KERNEL = {(0, 512, 128, "bf16"): "conv2 forward",
                (2, 64, 64, "bf16"): "wgrad3 (every width)",
                (2, 64, 256, "bf16"): "wgrad3s2 (stride 2)",
                (1, 256, 256, "bf16"): "conv2s2 data gradient",
                (0, 256, 128, "bf16"): "conv2s2f forward",
                (0, 64, 64, "bf16"): "conv64 forward",
                (0, 32, 64, "bf16"): "stem forward",
                (2, 32, 64, "bf16"): "stem weight gradient"}


def measured_traffic(workload, kernel):
    """HBM bytes per launch of `kernel` in `workload` from the committed
    counter summary, or None when there is none or the kernel's sources
    changed since the counters were taken (the summary records their
    SHA-256)."""
    import hashlib
    if kernel is None or workload not in TRAFFIC_PROFILE:
        return None
    try:
        text = open(TRAFFIC_PROFILE[workload]).read()
    except OSError:
        return None
    start = text.find("```json")
    if start < 0:
        return None
    table = json.loads(text[start + 7:text.index("```", start + 7)])
    entry = table.get(kernel)
    if entry is None:
        return None
    for path, digest in entry["sources"].items():
        with open(os.path.join(ROOT, path), "rb") as f:
            if hashlib.sha256(f.read()).hexdigest() != digest:
                return None
    return entry["bytes_per_launch"]


def step_flops_per_sample(hs, model):
    """Algorithmic FLOPs of one sample's forward and backward: 2 MACs forward,
    4 backward (data and weight gradient) for every layer except the first,
    whose input needs no data gradient (dense 3x3 taps)."""
    macs = hs.forward_macs(model)
    name, kind, shape, off = hs.param_table(model)[0]
    if kind == "conv_w":                    # first conv, stride 1 on 32x32 inputs
        first = 32 * 32 * shape[0] * shape[1] * shape[2] * shape[3]
    else:                                   # first linear layer
        first = shape[0] * shape[1]
    return 6 * macs - 2 * first


def percentile(v, q):
    s = sorted(v)
    k = (len(s) - 1) * q
    lo, hi = int(k), min(int(k) + 1, len(s) - 1)
    return s[lo] + (s[hi] - s[lo]) * (k - lo)


def timed_steps(tr, steps):
    """K steps, each bracketed by HIP events on the stream it runs on (the
    library orders all of a call's work on that stream); returns the per-step
    times (ms) and the wall time of the K steps (s)."""
    import torch
    main = torch.cuda.current_stream()
    ev = []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(main)
        tr.step()
        e1.record(main)
        ev.append((e0, e1))
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    return [e0.elapsed_time(e1) for e0, e1 in ev], wall


def probe_kernels(tr, dtype, steps=2):
    """Every GEMM family of the step, timed with HIP events around its launches
    (inside the library, on the stream each launch runs on): in the step as
    benchmarked (two streams), then with every launch on the caller's stream
    (no overlap).  Returns a list of dicts, largest time per step first."""
    from paper_2110_08941_amd import hs
    ws = tr.ws[0]
    peak = PEAK_TFLOPS[dtype]
    out = []
    for mode in (0, 1, 2):
        for bm, bn in PROBE_TILES:
            rec = {}
            for streams in (2, 1):
                hs.workspace_set_streams(ws, streams)
                hs.probe_enable(ws, mode, bm, bn, capacity=64 * steps)
                for _ in range(steps):
                    tr.step()
                tr.flush()
                ms, launches, flops = hs.probe_read(ws)
                rec[streams] = (ms, launches, flops)
            hs.probe_enable(ws, -1, 0, 0, 0)
            hs.workspace_set_streams(ws, 2)
            ms2, l2, f2 = rec[2]
            ms1, l1, f1 = rec[1]
            if l2 == 0:
                continue
            out.append({
                "kernel": kernel_name(mode, bm, bn, dtype), "mode": mode, "tile": [bm, bn],
                "launches_per_step": l2 / steps, "flops_per_step": f2 / steps,
                "ms_per_step": round(ms2 / steps, 4),
                "avg_launch_us": round(1e3 * ms2 / l2, 3),
                "frac_in_step": round(f2 / (ms2 * 1e-3) / 1e12 / peak, 4),
                "avg_launch_us_isolated": round(1e3 * ms1 / max(l1, 1), 3),
                "frac_isolated": round(f1 / (ms1 * 1e-3) / 1e12 / peak, 4) if ms1 > 0 else None})
    out.sort(key=lambda r: -r["ms_per_step"])
    return out


def run_workload(name, steps, warmup, seed, streams_mode=False, probe=True, single=False):
    """Warm-up, timed steps and per-kernel probes of one workload; returns the
    measurement dict and the trainer's last partition and losses."""
    import torch
    from paper_2110_08941_amd import hs
    from paper_2110_08941_amd.configs import WORKLOADS
    from paper_2110_08941_amd.driver import Trainer
    wl = WORKLOADS[name]
    tr = Trainer(wl, seed=seed, clock="measured" if streams_mode else "model",
                 steps=warmup + steps + (2 * 3 * len(PROBE_TILES) * 2 + 2 if probe else 0),
                 grouped=not streams_mode)
    try:
        if single and not streams_mode:
            hs.workspace_set_streams(tr.ws[0], 1)
        for _ in range(warmup):
            tr.step()
        tr.flush()
        torch.cuda.synchronize()
        tr.time_opt = True
        step_ms, wall = timed_steps(tr, steps)
        tr.time_opt = False
        tr.flush()
        opt_us = [1e3 * e0.elapsed_time(e1) for e0, e1 in tr.opt_events]
        opt_avg = sum(opt_us) / max(len(opt_us), 1)
        med = percentile(step_ms, 0.5)
        flops = step_flops_per_sample(hs, tr.model) * wl.total
        peak = PEAK_TFLOPS[wl.dtype]
        # simulated synchronous step time max_m X_m (Section 3): the measured
        # step time split over the workers in proportion to their partitions,
        # divided by each worker's simulated speed at that step
        sim = []
        for e in tr.log[warmup:warmup + steps]:
            share = [med * nm / float(wl.total) / s for nm, s in zip(e["n"], e["speed"])]
            sim.append(max(share))
        res = {
            "workload": name, "arch": wl.arch, "dtype": wl.dtype, "global_batch": wl.total,
            "workers": wl.workers, "steps": steps, "warmup": warmup,
            "samples_per_s": round(wl.total / (med * 1e-3), 2),
            "ms_per_step": round(med, 4),
            "ms_per_step_p10": round(percentile(step_ms, 0.1), 4),
            "ms_per_step_p90": round(percentile(step_ms, 0.9), 4),
            "ms_per_step_mean": round(sum(step_ms) / len(step_ms), 4),
            "wall_s": round(wall, 4),
            "step_roofline": {"bound": "mfma", "flops_per_step": flops,
                              "achieved": round(flops / (med * 1e-3) / 1e12, 2), "peak": peak,
                              "unit": "TFLOP/s",
                              "frac": round(flops / (med * 1e-3) / 1e12 / peak, 4)},
            "sim_step": {"max_m_X_m_ms_median": round(percentile(sim, 0.5), 4) if sim else None,
                         "definition": "model clock: step time x n_m / N / s_m, max over m"},
            "hbm_roofline": {"bound": "hbm",
                             "kernel": "wavg_sgd (fused partition-weighted average of %d fp32 "
                                       "gradients + %sSGD%s)"
                                       % (wl.workers, "momentum " if tr.mom is not None else "",
                                          " + bf16 copy" if tr.bf16 else ""),
                             "achieved": round(tr.opt_bytes() / (opt_avg * 1e-6) / 1e9, 1),
                             "peak": HBM_PEAK_GBS, "unit": "GB/s",
                             "frac": round(tr.opt_bytes() / (opt_avg * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
                             "traffic": measured_traffic(name, "wavg_sgd_kernel<2, true, true>"
                                                         if tr.bf16 and tr.mom is not None else None),
                             "bytes_per_launch": tr.opt_bytes(), "avg_launch_us": round(opt_avg, 3),
                             "launches": len(opt_us)},
        }
        if probe and not streams_mode and not single:
            res["kernels"] = probe_kernels(tr, wl.dtype)
        res["partitions_last"] = tr.log[-1]["n"] if tr.log else None
        res["loss_last"] = [round(v, 4) for v in tr.losses.cpu().tolist()]
    finally:
        tr.close()
    return res


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py measures one GPU: this build runs all simulated workers on a single "
              "MI355X and has no multi-GPU path (--gpus %d requested)" % args.gpus)
        sys.exit(2)
    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return
    from paper_2110_08941_amd.configs import WORKLOADS

    wl = WORKLOADS[args.workload]
    r = run_workload(args.workload, args.steps, args.warmup, args.seed, args.streams,
                     probe=not args.no_probe, single=args.single_stream)
    result = {
        "metric": METRIC.replace("ResNet-18", ARCH_NAME[wl.arch]),
        "value": r["samples_per_s"], "unit": "samples/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": r["ms_per_step"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": wl.dtype,
        "data": "synthetic",
        "config": {"workload": "%s: %s CIFAR-shape (3x32x32, 10 classes), N=%d over M=%d "
                               "workers, speeds %s%s, repartition every %s steps"
                               % (wl.name, wl.arch, wl.total, wl.workers, list(wl.speeds),
                                  " drifting (sigma %.2f)" % wl.drift_sigma if wl.drift_sigma else "",
                                  wl.window or "never"),
                   "global_batch": wl.total, "workers": wl.workers,
                   "parallelism": "simulated-dp%d-1gpu" % wl.workers,
                   "execution": "one stream per worker, measured clock" if args.streams
                   else "all workers in one pass per layer, model clock%s"
                   % (", every launch on one stream" if args.single_stream else "")},
        "timing": {"value_from": "N / median of the per-step HIP-event times",
                   "ms_per_step_p10": r["ms_per_step_p10"],
                   "ms_per_step_p90": r["ms_per_step_p90"],
                   "ms_per_step_mean": r["ms_per_step_mean"], "wall_s": r["wall_s"]},
        "step_roofline": r["step_roofline"],
    }
    kernels = r.get("kernels")
    if kernels:
        top = kernels[0]
        result["roofline"] = {
            "bound": "mfma", "kernel": top["kernel"],
            "achieved": round(top["frac_in_step"] * PEAK_TFLOPS[wl.dtype], 2),
            "peak": PEAK_TFLOPS[wl.dtype], "unit": "TFLOP/s", "frac": top["frac_in_step"],
            "frac_isolated": top["frac_isolated"],
            "traffic": measured_traffic(args.workload,
                                        PROBE_KERNEL.get((top["mode"], top["tile"][0],
                                                          top["tile"][1], wl.dtype))),
            "avg_launch_us": top["avg_launch_us"], "launches_per_step": top["launches_per_step"],
            "flops_per_launch": top["flops_per_step"] / max(top["launches_per_step"], 1),
            "selection": "the GEMM family with the largest time per step (HIP events "
                         "around its launches in the step)"}
        for k in kernels:   # counted HBM bytes per launch, where the summary has the family
            k["traffic"] = measured_traffic(args.workload, PROBE_KERNEL.get(
                (k["mode"], k["tile"][0], k["tile"][1], wl.dtype)))
        result["kernels"] = kernels
    result["hbm_roofline"] = r["hbm_roofline"]
    result["sim_step"] = r["sim_step"]
    result["partitions_last"] = r["partitions_last"]
    result["loss_last"] = r["loss_last"]
    result["wavg_sgd_standalone"] = standalone_wavg()
    if not args.no_probe:    # the attainable rates are probes too
        result["attainable"] = attainable()
    if "attainable" in result and wl.dtype == "bf16":   # the loop runs bf16 MFMAs
        mf = result["attainable"]["mfma_bf16_loop"]["achieved"]
        if "roofline" in result:
            result["roofline"]["frac_of_attainable"] = round(result["roofline"]["achieved"] / mf, 4)
        result["step_roofline"]["frac_of_attainable"] = round(
            result["step_roofline"]["achieved"] / mf, 4)
    if "attainable" in result:
        result["hbm_roofline"]["frac_of_attainable"] = round(
            result["hbm_roofline"]["achieved"] / result["attainable"]["copy_1GiB"]["achieved"], 4)
    if not args.no_extra and not args.streams:
        extra = {}
        for name in EXTRA:
            if name == args.workload:
                continue
            e = run_workload(name, 10, 3, args.seed, probe=not args.no_probe)
            k = e.pop("kernels", None)
            if k:
                e["top_kernels"] = k[:4]
            extra[name] = e
        result["other_workloads"] = extra
    if not args.no_cpu_baseline:
        samples = args.cpu_samples or CPU_SAMPLES.get(wl.arch, 64)
        result["cpu_baseline"] = cpu_baseline(wl, args.seed, samples)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
