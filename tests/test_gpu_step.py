"""GPU parity of whole steps (workers on their streams + fused weighted
average + SGD + repartition) against the oracle, and of the partition
sequence over many steps (bit-exact replay of the logged worker times)."""
import dataclasses

import numpy as np
import pytest
import torch

from oracle import models as Mo
from oracle import step as S
from paper_2110_08941_amd import synth
from paper_2110_08941_amd.configs import WORKLOADS
from tests.gpu_util import require_gpu, normwise, log

pytestmark = pytest.mark.gpu

TOL = {"fp32": 1e-4, "bf16": 2e-2}
STORAGE = {"fp32": "exact", "bf16": "bf16"}


def make_trainer(name, total=None, steps=None, clock="model", separated=False, seed=0, **kw):
    require_gpu()
    from paper_2110_08941_amd.driver import Trainer
    wl = WORKLOADS[name]
    if total is not None:
        wl = dataclasses.replace(wl, total=total)
    net = Mo.build(wl.arch)
    table, P = Mo.param_table(net)
    theta = synth.he_normal(table, P, seed)
    if separated:
        theta = synth.separate_decisions(table, theta, seed)
    tr = Trainer(wl, seed=seed, clock=clock, steps=steps, theta0=theta, **kw)
    return tr, net, theta


@pytest.mark.parametrize("grouped", [False, True])
@pytest.mark.parametrize("name,total,separated", [
    ("mlp_fp32", 256, False),            # the full MLP workload
    ("smallcnn_fp32", 40, False),
    ("resnet18_fp32", 24, True),
    ("resnet18_bf16", 32, True),
    ("resnet50_bf16", 24, True),
    ("vgg16_bf16", 32, True)])
def test_one_step(name, total, separated, grouped):
    """theta' - theta after one step (worker gradients -- on their own streams,
    or all in one pass -- weighted average, momentum SGD) against the oracle's
    step on the same partition."""
    log("one step %s N=%d grouped=%s" % (name, total, grouped))
    tr, net, theta = make_trainer(name, total=total, steps=1, separated=separated,
                                  grouped=grouped)
    try:
        n = tr.part.partition()
        x, y = tr.batch(0)
        xs, ys = x.cpu().numpy(), y.cpu().numpy()
        tr.step()
        torch.cuda.synchronize()
        got = tr.theta.cpu().numpy().astype(np.float64)
        gpu_losses = tr.losses.cpu().numpy()
    finally:
        tr.close()
    wl = tr.wl
    st = STORAGE[wl.dtype]
    out = S.step(lambda th, xm, ym: Mo.worker_grad(net, th, xm, ym, storage=st),
                 theta.astype(np.float64), None, xs, ys, n, wl.lr, wl.mu, wl.wd)
    d_ref = out["theta"] - theta
    err = normwise(got - theta, d_ref)
    log("  partition %s  normwise update err %.3e" % (n, err))
    assert err <= TOL[wl.dtype]
    assert normwise(got, out["theta"]) <= TOL[wl.dtype]
    np.testing.assert_allclose(gpu_losses, out["losses"], rtol=TOL[wl.dtype], atol=0)


def replay(log_entries, M, N, window):
    """Partition sequence of Algorithm 1 from logged (tau, speed): even start,
    then every `window` steps CP = n / mean(tau / speed), repartition."""
    n = S.even_split(M, N)
    seq, xsum = [], [0.0] * M
    for t, e in enumerate(log_entries):
        seq.append(list(n))
        for j in range(M):
            xsum[j] = xsum[j] + float(e["tau"][j]) / float(e["speed"][j])
        if (t + 1) % window == 0:
            n = S.repartition(S.estimate_cp(n, [v / float(window) for v in xsum]), N)
            xsum = [0.0] * M
    return seq


@pytest.mark.parametrize("name,steps", [("smallcnn_fp32", 20), ("resnet18_bf16", 40)])
def test_partition_sequence_replays_bit_exact(name, steps):
    """Measured clock: the partitions the GPU run used, step by step, equal
    the oracle's Algorithm 1 replayed on the logged times and speeds (the
    times are hardware-dependent; their repartition is not)."""
    log("partition replay %s %d steps" % (name, steps))
    tr, _, _ = make_trainer(name, steps=steps, clock="measured")
    try:
        tr.run(steps)
        entries = tr.log
        wl = tr.wl
    finally:
        tr.close()
    used = [e["n"] for e in entries]
    assert len(used) == steps
    assert used == replay(entries, wl.workers, wl.total, wl.window)
    assert all(sum(n) == wl.total and min(n) >= 1 for n in used)
    log("  partitions at window starts: %s" % [used[t] for t in range(0, steps, wl.window)])
    # the partitions follow the speeds: the fastest worker gets the most data
    last = used[-1]
    speed = entries[-1]["speed"]
    assert int(np.argmax(last)) == int(np.argmax(speed)) or wl.drift_sigma > 0


@pytest.mark.parametrize("grouped", [False, True])
def test_model_clock_partitions(grouped):
    """Model clock (X_m = n_m / s_m): even split for the first window, then
    exactly proportional to the speeds 1:1:2:4 (64/64/128/256 of 512)."""
    tr, _, _ = make_trainer("smallcnn_fp32", steps=10, clock="model", grouped=grouped)
    try:
        tr.run(10)
        used = [e["n"] for e in tr.log]
    finally:
        tr.close()
    assert used[:5] == [[128] * 4] * 5
    assert used[5:] == [[64, 64, 128, 256]] * 5


@pytest.mark.parametrize("grouped", [False, True])
def test_multistep_theta_small_cnn(grouped):
    """Ten steps of the small CNN workload (reduced to N = 32, repartition
    every 5 steps with the model clock) against the oracle's driver."""
    log("multistep small cnn grouped=%s" % grouped)
    wl = dataclasses.replace(WORKLOADS["smallcnn_fp32"], total=32, window=5, steps=10)
    require_gpu()
    from paper_2110_08941_amd.driver import Trainer
    net = Mo.build(wl.arch)
    table, P = Mo.param_table(net)
    theta = synth.he_normal(table, P, 0)
    tr = Trainer(wl, seed=0, clock="model", steps=10, theta0=theta, n_batches=10,
                 grouped=grouped)
    try:
        batches = [(x.cpu().numpy(), y.cpu().numpy()) for x, y in tr.batches]
        tr.run(10)
        got = tr.theta.cpu().numpy().astype(np.float64)
        used = [e["n"] for e in tr.log]
        speeds = tr.speeds
    finally:
        tr.close()
    out = S.run(lambda th, xm, ym: Mo.worker_grad(net, th, xm, ym), theta.astype(np.float64),
                batches, speeds, wl.window, wl.lr, wl.mu, wl.wd)
    assert used == out["partitions"]
    err = normwise(got - theta, out["theta"] - theta)
    log("  partitions %s ... %s, normwise err %.3e" % (used[0], used[-1], err))
    assert err <= TOL["fp32"]


@pytest.mark.parametrize("grouped", [False, True])
@pytest.mark.parametrize("name", ["resnet18_bf16", "resnet50_bf16"])
def test_multistep_theta_bf16_resnet(name, grouped):
    """Four steps of a bf16 ResNet workload (N = 24 over its 8 workers,
    separated decisions, lr 0.01 so that they stay separated, momentum and
    weight decay) on one workspace per worker: the later calls take the
    packed weights prepared on the second stream and run the weight
    gradients there.  The update theta_4 - theta_0 against the oracle's
    driver with bf16 storage, within the bf16 bar."""
    log("multistep %s grouped=%s" % (name, grouped))
    wl = dataclasses.replace(WORKLOADS[name], total=24, steps=4, drift_sigma=0.0, lr=0.01)
    require_gpu()
    from paper_2110_08941_amd.driver import Trainer
    net = Mo.build(wl.arch)
    table, P = Mo.param_table(net)
    theta = synth.separate_decisions(table, synth.he_normal(table, P, 2), 2)
    tr = Trainer(wl, seed=2, clock="model", steps=4, theta0=theta, n_batches=4, grouped=grouped)
    try:
        batches = [(x.cpu().numpy(), y.cpu().numpy()) for x, y in tr.batches]
        tr.run(4)
        got = tr.theta.cpu().numpy().astype(np.float64)
        used = [e["n"] for e in tr.log]
        speeds = tr.speeds
    finally:
        tr.close()
    out = S.run(lambda th, xm, ym: Mo.worker_grad(net, th, xm, ym, storage="bf16"),
                theta.astype(np.float64), batches, speeds, wl.window, wl.lr, wl.mu, wl.wd)
    assert used == out["partitions"]
    err = normwise(got - theta, out["theta"] - theta)
    log("  partitions %s, normwise err of the update %.3e" % (used[0], err))
    assert err <= TOL["bf16"]


MODES = {
    # Sync-SGD: even split throughout, plain mean
    "sync": dict(window=0, exchange="mean"),
    # Dynamic Partitioning without the enhancement: plain mean
    "dp_mean": dict(window=2, exchange="mean"),
    # EDP with an EMA estimator and cosine annealing
    "edp_ema_cosine": dict(window=2, exchange="edp", estimator=("ema", 0.5),
                           lr_schedule=("cosine", 10, 0.001)),
    # EDP with the mean of the last 3 windows' estimates
    "edp_history": dict(window=2, exchange="edp", estimator=("history", 3)),
}


@pytest.mark.parametrize("grouped", [False, True])
@pytest.mark.parametrize("mode", sorted(MODES))
def test_multistep_modes_small_cnn(mode, grouped):
    """Ten steps of the small CNN (N = 32, 4 workers at speeds 1:1:2:4, an
    additive delay on workers 0 and 2, model clock) in each exchange /
    partitioning / estimator / schedule mode against the oracle's driver:
    partitions and batch times bit-exact, theta within the fp32 bar."""
    cfg = dict(MODES[mode])
    window = cfg.pop("window")
    log("multistep mode=%s grouped=%s" % (mode, grouped))
    wl = dataclasses.replace(WORKLOADS["smallcnn_fp32"], total=32, window=window, steps=10,
                             mu=0.9, wd=5e-4)
    require_gpu()
    from paper_2110_08941_amd.driver import Trainer
    net = Mo.build(wl.arch)
    table, P = Mo.param_table(net)
    theta = synth.he_normal(table, P, 0)
    delays = [3.0, 0.0, 1.5, 0.0]
    tr = Trainer(wl, seed=0, clock="model", steps=10, theta0=theta, n_batches=10,
                 grouped=grouped, delays=delays, **cfg)
    try:
        batches = [(x.cpu().numpy(), y.cpu().numpy()) for x, y in tr.batches]
        tr.run(10)
        got = tr.theta.cpu().numpy().astype(np.float64)
        used = [e["n"] for e in tr.log]
        xs = [e["x"] for e in tr.log]
        speeds = tr.speeds
    finally:
        tr.close()
    sched = cfg.get("lr_schedule")
    out = S.run(lambda th, xm, ym: Mo.worker_grad(net, th, xm, ym), theta.astype(np.float64),
                batches, speeds, window, wl.lr, wl.mu, wl.wd, exchange=cfg["exchange"],
                delays=delays, estimator=cfg.get("estimator", ("window",)),
                lr_total=sched[1] if sched else None, lr_min=sched[2] if sched else 0.0)
    assert used == out["partitions"]
    assert xs == out["xs"]
    if window == 0:
        assert used == [[8, 8, 8, 8]] * 10
    else:
        assert used[-1] != [8, 8, 8, 8]
    err = normwise(got - theta, out["theta"] - theta)
    log("  partitions %s ... %s, normwise err %.3e" % (used[0], used[-1], err))
    assert err <= TOL["fp32"]


def test_full_size_weighted_average_invariant():
    """At the full small-CNN size (N = 512, workers 1:1:2:4): the partition
    -weighted average of the GPU worker gradients equals the GPU gradient of
    the whole batch computed by a single worker (the network has no
    batch-norm, so Eq. (1) with weights n_m / N gives the full-batch mean)."""
    hs = require_gpu()
    log("full-size invariant small cnn")
    tr, _, _ = make_trainer("smallcnn_fp32", steps=1, clock="model")
    try:
        n = hs.repartition([1.0, 1.0, 2.0, 4.0], tr.N)
        x, y = tr.batch(0)
        tr.launch_workers(n, x, y, timed=False)
        gbar = torch.empty(tr.P, device="cuda")
        hs.weighted_average([g.data_ptr() for g in tr.grads], n, tr.P, gbar.data_ptr())
        full = torch.empty(tr.P, device="cuda")
        ws = hs.workspace_create(tr.model, tr.N)
        hs.worker_grad(tr.model, ws, tr.theta.data_ptr(), 0, x.data_ptr(), y.data_ptr(), tr.N,
                       full.data_ptr(), 0, 0)
        torch.cuda.synchronize()
        hs.workspace_destroy(ws)
        err = normwise(gbar.cpu().numpy(), full.cpu().numpy())
    finally:
        tr.close()
    log("  partition %s normwise err %.3e" % (n, err))
    assert err <= TOL["fp32"]
