"""Benchmark of the heterogeneous data-parallel training step on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload resnet18_bf16]
                    [--no-cpu-baseline] [--gpus 1]

One step = every simulated worker's forward+backward on its partition of a
synthetic CIFAR-shaped batch, the fused partition-weighted gradient average +
momentum SGD, and -- at the end of every repartition window -- the
compute-power estimate and the repartition of the next window.  By default
all workers run in one pass over the layers (hs_workers_grad: each layer is
launched once over the whole batch, with per-worker batch-norm statistics,
losses and weight gradients) and worker times follow the model clock
X_m = n_m / s_m; --streams runs one hs_worker_grad per worker on its own HIP
stream with event-measured times instead.  W untimed steps, then K timed
steps between two device synchronisations; the batches are resident in HBM
before timing.

Prints ONE JSON line: samples/s over the K steps, the roofline position of
the dominant GEMM kernel (timed live with HIP events on the stream it runs on
during the timed steps), the HBM roofline position of the fused weighted
average + SGD launch of every timed step (event-timed on the main stream),
the same kernel alone on 8 fp32 buffers of 25M elements, and the CPU oracle's
throughput on a bounded sample of the same step, timed on this host.
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

# GEMM kernel probed for the roofline (mode, bm, bn), per workload: the
# implicit-GEMM kernel that takes the largest share of the step's time (mode 0
# forward, 1 data gradient, 2 weight gradient; bm = 512 selects the 32x32x16
# MFMA forward / data-gradient kernel with 512-row tiles, bm = bn = 64 in mode
# 2 the patch weight-gradient kernel).
PROBE = {"resnet18_bf16": (0, 512, 128), "resnet18_fp32": (2, 128, 128),
         "resnet50_bf16": (0, 512, 128),
         "vgg16_bf16": (0, 512, 128), "smallcnn_fp32": (2, 128, 128), "mlp_fp32": (0, 128, 64)}
MODE_NAME = {0: "forward", 1: "data gradient", 2: "weight gradient"}
# template instance of each probed kernel whose HBM traffic has been counted
PROBE_KERNEL = {(0, 512, 128, "bf16"): "conv2_kernel<0, 128, 9, 0, true>"}


def kernel_name(mode, bm, bn, dtype):
    if bm == 512:
        return "conv2_kernel<%s, %dx%d tile, 32x32x16 MFMA, %s>" % (MODE_NAME[mode], bm, bn, dtype)
    if mode == 2 and bm == 64 and bn == 64 and dtype == "bf16":
        return "wgrad3_kernel<3x3 weight gradient, 64x64x9 tile, %s>" % dtype
    return "igemm_fast_kernel<%s, mode %d (%s), %dx%d tile>" % (dtype, mode, MODE_NAME[mode], bm, bn)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="resnet18_bf16")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-samples", type=int, default=None,
                    help="samples of the CPU oracle's bounded step (default: about 15 s of "
                         "host work for the workload's network)")
    ap.add_argument("--streams", action="store_true",
                    help="one stream per worker, measured clock (default: one pass)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB four times (the reference "
                         "kernel that scales the FETCH_SIZE / WRITE_SIZE counters to bytes)")
    ap.add_argument("--probe", default=None,
                    help="GEMM instantiation timed for the roofline, as mode,bm,bn")
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
        threads = 1
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
    return {"value": round(sum(n) / dt, 3), "unit": "samples/s", "cores": int(threads),
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


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py measures one GPU: this build runs all simulated workers on a single "
              "MI355X and has no multi-GPU path (--gpus %d requested)" % args.gpus)
        sys.exit(2)
    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return
    import torch
    from paper_2110_08941_amd import hs
    from paper_2110_08941_amd.configs import WORKLOADS
    from paper_2110_08941_amd.driver import Trainer

    wl = WORKLOADS[args.workload]
    tr = Trainer(wl, seed=args.seed, clock="measured" if args.streams else "model",
                 steps=args.warmup + args.steps, grouped=not args.streams)
    mode, bm, bn = (PROBE[args.workload] if args.probe is None
                    else tuple(int(v) for v in args.probe.split(",")))
    for w in tr.ws:
        hs.probe_enable(w, mode, bm, bn, capacity=64 * (args.steps + 1))
    for _ in range(args.warmup):
        tr.step()
    tr.flush()
    torch.cuda.synchronize()
    for w in tr.ws:
        hs.probe_read(w)                    # drop the warm-up launches
    tr.time_opt = True
    t0 = time.perf_counter()
    for _ in range(args.steps):
        tr.step()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    tr.time_opt = False
    opt_us = [1e3 * e0.elapsed_time(e1) for e0, e1 in tr.opt_events]
    opt_avg = sum(opt_us) / max(len(opt_us), 1)
    tr.flush()
    ms, launches, flops = 0.0, 0, 0.0
    for w in tr.ws:
        a, b, c = hs.probe_read(w)
        ms, launches, flops = ms + a, launches + b, flops + c
    value = wl.total * args.steps / elapsed
    achieved = flops / (ms * 1e-3) / 1e12 if ms > 0 else 0.0
    peak = PEAK_TFLOPS[wl.dtype]
    loss = tr.losses.cpu().tolist()
    parts = [e["n"] for e in tr.log]
    result = {
        "metric": METRIC.replace("ResNet-18", ARCH_NAME[wl.arch]), "value": round(value, 2), "unit": "samples/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(1e3 * elapsed / args.steps, 3), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": wl.dtype, "data": "synthetic",
        "config": {"workload": "%s: %s CIFAR-shape (3x32x32, 10 classes), N=%d over M=%d "
                               "workers, speeds %s%s, repartition every %s steps"
                               % (wl.name, wl.arch, wl.total, wl.workers, list(wl.speeds),
                                  " drifting (sigma %.2f)" % wl.drift_sigma if wl.drift_sigma else "",
                                  wl.window or "never"),
                   "global_batch": wl.total, "workers": wl.workers,
                   "parallelism": "simulated-dp%d-1gpu" % wl.workers,
                   "execution": "one stream per worker, measured clock" if args.streams
                   else "all workers in one pass per layer, model clock"},
        "roofline": {"bound": "mfma", "kernel": kernel_name(mode, bm, bn, wl.dtype),
                     "achieved": round(achieved, 2), "peak": peak, "unit": "TFLOP/s",
                     "frac": round(achieved / peak, 4),
                     "traffic": measured_traffic(args.workload,
                                                 PROBE_KERNEL.get((mode, bm, bn, wl.dtype))),
                     "launches": launches, "avg_launch_us": round(1e3 * ms / max(launches, 1), 3),
                     "flops_per_launch": flops / max(launches, 1)},
        "hbm_roofline": {"bound": "hbm", "kernel": "wavg_sgd (fused partition-weighted average of "
                                                   "%d fp32 gradients + momentum SGD%s)"
                                                   % (wl.workers, " + bf16 copy" if tr.bf16 else ""),
                         "achieved": round(tr.opt_bytes() / (opt_avg * 1e-6) / 1e9, 1),
                         "peak": HBM_PEAK_GBS, "unit": "GB/s",
                         "frac": round(tr.opt_bytes() / (opt_avg * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
                         "traffic": measured_traffic(args.workload,
                                                     "wavg_sgd_kernel<2, true, true>"
                                                     if tr.bf16 and tr.mom is not None else None),
                         "bytes_per_launch": tr.opt_bytes(), "avg_launch_us": round(opt_avg, 3),
                         "launches": len(opt_us)},
        "partitions_last": parts[-1] if parts else None,
        "loss_last": [round(v, 4) for v in loss],
    }
    tr.close()
    result["wavg_sgd_standalone"] = standalone_wavg()
    if not args.no_cpu_baseline:
        samples = args.cpu_samples or CPU_SAMPLES.get(wl.arch, 64)
        result["cpu_baseline"] = cpu_baseline(wl, args.seed, samples)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
