"""Sync-SGD, DP-SGD and EDP-SGD side by side on one GPU with synthetic data
(the comparison of Section 5).

Heterogeneity is simulated the way Section 5 does it: a fixed time delay is
added to every mini-batch of a subset of the workers (by default the first
half), sized as a fraction of the mean mini-batch time of the even split
(0.25 is the paper's low level, 0.5 its high level).  Every mode starts from
the same parameters and sees the same batches:

  sync  the even split throughout and the plain mean of the gradients;
  dp    Dynamic Partitioning (Algorithm 1) with the plain mean;
  edp   Dynamic Partitioning with the partition-weighted average (Section 4.2).

For every step the report holds the simulated batch time of each worker,
X_m = tau_m / s_m + delay_m, and the step time max_m X_m (the slowest worker
sets the pace of a synchronous step, Section 3).  Per mode it gives the
histogram of each worker's X_m (the batch-time histograms with and without
Dynamic Partitioning), the mean of max_m X_m, and each worker's split of the
step time into its own batch time and the wait for the slowest (the time
breakdown of the AWS case study).  The mean training loss per step is
reported too (synthetic labels: it shows that all modes train, nothing
about accuracy).

clock="model" takes tau_m = n_m (time in sample units, independent of the
hardware); clock="measured" takes tau_m from HIP events around each worker's
gradient (milliseconds), with the workers run one after another on one
stream so that each time is that worker's work alone, as if it had a device
of its own.

    python -m paper_2110_08941_amd.compare --workload resnet18_bf16 --steps 60 \\
        --clock measured --delay-frac 0.5 --out report.json
"""
import argparse
import dataclasses
import json
import sys

import numpy as np

MODES = {
    "sync": dict(window=0, exchange="mean"),
    "dp": dict(window=None, exchange="mean"),
    "edp": dict(window=None, exchange="edp"),
}


def delay_vector(m, delayed, delay):
    """Per-worker additive delay: `delay` on the workers listed in `delayed`."""
    d = [0.0] * m
    for j in delayed:
        if not 0 <= j < m:
            raise ValueError("delayed worker %d out of range" % j)
        d[j] = float(delay)
    return d


def summarize(xs, edges, skip=0):
    """Batch-time statistics of one run.  xs[t][m] = X_m at step t; the first
    `skip` steps are left out.  Histograms use the given bin edges (shared by
    the modes, so that they are comparable); values outside fall in the end
    bins."""
    x = np.asarray(xs, dtype=np.float64)[skip:]
    if x.ndim != 2 or x.shape[0] == 0:
        raise ValueError("need at least one step after the skipped ones")
    edges = np.asarray(edges, dtype=np.float64)
    step = x.max(axis=1)
    wait = step[:, None] - x
    clipped = np.clip(x, edges[0], edges[-1])
    hist = [np.histogram(clipped[:, j], edges)[0].tolist() for j in range(x.shape[1])]
    return {
        "steps": int(x.shape[0]),
        "max_x_mean": float(step.mean()),
        "max_x_max": float(step.max()),
        "sim_time": float(step.sum()),
        "x_mean": x.mean(axis=0).tolist(),
        "x_std": x.std(axis=0).tolist(),
        "wait_mean": wait.mean(axis=0).tolist(),
        "wait_frac": (wait.sum(axis=0) / step.sum()).tolist(),
        "spread_mean": float((x.max(axis=1) - x.min(axis=1)).mean()),
        "hist": hist,
    }


def shared_edges(runs, bins, skip=0):
    lo = min(float(np.min(np.asarray(r)[skip:])) for r in runs)
    hi = max(float(np.max(np.asarray(r)[skip:])) for r in runs)
    if hi <= lo:
        hi = lo + 1.0
    return np.linspace(lo, hi, bins + 1)


def render(name, summ, edges, width=40):
    """Text histogram of every worker's batch time."""
    lines = ["%s: mean max_m X_m %.4g, worker X_m mean %s" %
             (name, summ["max_x_mean"], " ".join("%.3g" % v for v in summ["x_mean"]))]
    top = max(max(h) for h in summ["hist"]) or 1
    for j, h in enumerate(summ["hist"]):
        for b, c in enumerate(h):
            if c:
                lines.append("  w%-2d [%9.4g, %9.4g) %5d %s" % (j, edges[b], edges[b + 1], c,
                                                                "#" * max(1, c * width // top)))
    return "\n".join(lines)


def run_mode(wl, mode, steps, seed, clock, delays, estimator, lr_schedule, theta0):
    import torch
    from .driver import Trainer
    cfg = MODES[mode]
    w = dataclasses.replace(wl, window=wl.window if cfg["window"] is None else cfg["window"],
                            steps=steps)
    tr = Trainer(w, seed=seed, clock=clock, steps=steps, theta0=theta0, grouped=False,
                 exchange=cfg["exchange"], delays=delays, estimator=estimator,
                 lr_schedule=lr_schedule, serial=(clock == "measured"))
    losses = []
    try:
        for _ in range(steps):
            n = tr.step()
            nn = torch.tensor(n, dtype=torch.float32, device=tr.dev)
            losses.append((tr.losses * nn).sum() / float(sum(n)))
        tr.flush()
        loss = torch.stack(losses).cpu().tolist()
        log = tr.log
    finally:
        tr.close()
    return {"x": [e["x"] for e in log], "partitions": [e["n"] for e in log], "loss": loss}


def calibrate(wl, steps, seed, clock, theta0):
    """Mean batch time of the even split without delays (the unit the delays
    are sized in).  Model clock: mean of (N/M) / s_m; measured: a short run."""
    if clock == "model":
        n = wl.total / float(wl.workers)
        return float(np.mean([n / s for s in wl.speeds]))
    r = run_mode(wl, "sync", steps, seed, clock, None, ("window",), None, theta0)
    return float(np.mean(np.asarray(r["x"])[1:]))


def main(argv=None):
    from .configs import WORKLOADS
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--workload", default="resnet18_bf16", choices=sorted(WORKLOADS))
    ap.add_argument("--steps", type=int, default=60)
    ap.add_argument("--window", type=int, default=None, help="repartition period (default: the workload's)")
    ap.add_argument("--clock", choices=("model", "measured"), default="model")
    ap.add_argument("--delay-frac", type=float, default=0.5,
                    help="delay as a fraction of the mean even-split batch time")
    ap.add_argument("--delayed", default=None, help="comma-separated delayed workers (default: first half)")
    ap.add_argument("--hetero-speeds", action="store_true",
                    help="keep the workload's speed ratios (default: equal speeds, delays only)")
    ap.add_argument("--estimator", default="window", help="window | ema:ALPHA | history:H")
    ap.add_argument("--cosine", action="store_true", help="cosine-annealed learning rate over the run")
    ap.add_argument("--modes", default="sync,dp,edp")
    ap.add_argument("--bins", type=int, default=16)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--out", default=None, help="write the full report (with per-step traces) as JSON")
    a = ap.parse_args(argv)

    wl = WORKLOADS[a.workload]
    m = wl.workers
    wl = dataclasses.replace(wl, drift_sigma=0.0, start_even=True,
                             window=a.window if a.window is not None else max(wl.window, 1))
    if not a.hetero_speeds:
        wl = dataclasses.replace(wl, speeds=(1.0,) * m)
    delayed = (list(range(m // 2)) if a.delayed is None
               else [int(v) for v in a.delayed.split(",") if v != ""])
    est = a.estimator.split(":")
    estimator = (("window",) if est[0] == "window" else
                 ("ema", float(est[1])) if est[0] == "ema" else ("history", int(est[1])))
    lr_schedule = ("cosine", a.steps, 0.0) if a.cosine else None
    modes = [v for v in a.modes.split(",") if v]
    for v in modes:
        if v not in MODES:
            raise SystemExit("unknown mode %r" % v)

    base = calibrate(wl, min(a.steps, 6), a.seed, a.clock, None)
    delay = a.delay_frac * base
    delays = delay_vector(m, delayed, delay)
    runs = {v: run_mode(wl, v, a.steps, a.seed, a.clock, delays, estimator, lr_schedule, None)
            for v in modes}
    skip = 1 if a.clock == "measured" else 0         # the first step carries start-up costs
    edges = shared_edges([r["x"] for r in runs.values()], a.bins, skip)
    report = {"workload": a.workload, "clock": a.clock,
              "unit": "ms" if a.clock == "measured" else "samples / speed",
              "workers": m, "speeds": list(wl.speeds), "window": wl.window,
              "estimator": list(estimator), "even_split_batch_time": base,
              "delay": delay, "delayed": delayed, "steps": a.steps, "skip": skip,
              "edges": edges.tolist(), "modes": {}}
    for v, r in runs.items():
        summ = summarize(r["x"], edges, skip)
        summ["final_partition"] = r["partitions"][-1]
        summ["loss_first"], summ["loss_last"] = r["loss"][0], r["loss"][-1]
        report["modes"][v] = summ
        print(render(v, summ, edges), file=sys.stderr)
    if "sync" in runs:
        ref = report["modes"]["sync"]["max_x_mean"]
        for v in modes:
            report["modes"][v]["speedup_vs_sync"] = ref / report["modes"][v]["max_x_mean"]
    if a.out:
        full = dict(report, traces={v: r for v, r in runs.items()})
        with open(a.out, "w") as f:
            json.dump(full, f)
    print(json.dumps(report))
    return 0


if __name__ == "__main__":
    sys.exit(main())
