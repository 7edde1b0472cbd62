"""GPU parity of hs_workers_grad: all workers' gradients in one pass over the
layers (each layer launched once over the whole batch; batch-norm statistics,
losses and weight gradients per worker), checked worker by worker against the
exact oracle, and against separate hs_worker_grad calls.

Error measure, tolerances and decision regimes are those of
test_gpu_worker.py: per parameter tensor against the exact float64 oracle,
1e-4 (fp32) / 2e-2 (bf16), or 3 x the oracle's own error at the path's
precision on a tensor where that floor exceeds the bar.  The workload
configurations are checked at their own sizes against stored oracle values
(tests/fullsize.py) on sampled entries, each tensor's floor being the
oracle's own error over all its entries: every worker of the ResNet-18 bf16
(N = 2048) and fp32 (N = 1024) workloads, the smallest and the largest worker
of the VGG-16 workload (N = 4096), every worker of the small-CNN workload
(N = 512), the two smallest of ResNet-50 (N = 1024).  Every case prints its
name before it runs."""
import os

import numpy as np
import pytest
import torch

from oracle import models as Mo
from paper_2110_08941_amd import synth
from paper_2110_08941_amd.configs import WORKLOADS
from tests import fullsize as F
from tests.gpu_util import (require_gpu, log, TOL, FLOOR_FACTOR, pertensor, check_pertensor,
                            separate_by_bias, oracle_floor)
from tests.test_gpu_worker import decision_aware, check_padding, AMBIGUOUS

pytestmark = pytest.mark.gpu


def in_shape(arch):
    return (784,) if arch == "mlp" else (3, 32, 32)


def run_workers(arch, dtype, n, theta, x, y, separate=False):
    """Per-worker gradients and losses from one hs_workers_grad call (or, with
    separate=True, from one hs_worker_grad call per worker)."""
    hs = require_gpu()
    m = hs.model_create(arch, dtype)
    try:
        P = hs.num_params(m)
        th = torch.from_numpy(np.asarray(theta, dtype=np.float32)).cuda()
        tb = None
        if dtype == "bf16":
            tb = torch.empty(P, dtype=torch.int16, device="cuda")
            hs.params_to_bf16(th.data_ptr(), tb.data_ptr(), P)
        xd, yd = torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda()
        grads = [torch.full((P,), float("nan"), device="cuda") for _ in n]
        loss = torch.zeros(len(n), device="cuda")
        tbp = tb.data_ptr() if tb is not None else 0
        if separate:
            ws = hs.workspace_create(m, max(n))
            o, ew = 0, xd.element_size() * int(np.prod(in_shape(arch)))
            for i, nm in enumerate(n):
                hs.worker_grad(m, ws, th.data_ptr(), tbp, xd.data_ptr() + o * ew,
                               yd.data_ptr() + o * 4, nm, grads[i].data_ptr(),
                               loss.data_ptr() + 4 * i, 0)
                o += nm
        else:
            ws = hs.workspace_create(m, sum(n))
            hs.workers_grad(m, ws, th.data_ptr(), tbp, xd.data_ptr(), yd.data_ptr(), n,
                            [g.data_ptr() for g in grads], loss.data_ptr(), 0)
        torch.cuda.synchronize()
        hs.workspace_destroy(ws)
        return [g.cpu().numpy() for g in grads], loss.cpu().numpy()
    finally:
        hs.model_destroy(m)


def slices(n):
    o = np.concatenate([[0], np.cumsum(n)]).astype(int)
    return [(int(o[i]), int(o[i + 1])) for i in range(len(n))]


HE_INIT = [("mlp", "fp32", [1, 7, 3]), ("mlp", "bf16", [5, 11]),
           ("small_cnn", "fp32", [2, 1, 5, 3]),
           ("small_cnn", "fp32", [1] * 16),
           ("small_cnn", "fp32", [1, 2, 1, 3, 1, 1, 2, 1, 1, 1, 4, 1, 1, 2, 1, 3])]


@pytest.mark.parametrize("arch,dtype,n", HE_INIT)
def test_workers_grad_he_init(arch, dtype, n):
    """BN-free networks at He init: every worker's gradient and loss against
    the exact oracle on that worker's rows (decision-aware), per tensor."""
    log("workers_grad he-init %s %s n=%s" % (arch, dtype, n))
    net = Mo.build(arch)
    table, P = Mo.param_table(net)
    theta = synth.he_normal(table, P, len(n))
    x, y = synth.batch(in_shape(arch), sum(n), len(n), 1)
    grads, losses = run_workers(arch, dtype, n, theta, x, y)
    for i, (a, b) in enumerate(slices(n)):
        g = grads[i]
        assert np.all(np.isfinite(g)), "worker %d: non-finite gradient" % i
        check_padding(arch, g)
        ref, namb, flips, ref_loss = decision_aware(net, theta, x[a:b], y[a:b], g,
                                                    AMBIGUOUS[dtype])
        log("  worker %d (n=%d): ambiguous %d, flipped %d, loss %.6f vs %.6f"
            % (i, b - a, namb, flips, losses[i], ref_loss))
        check_pertensor(g, ref, table, TOL[dtype], what="worker %d vs exact" % i)
        assert abs(losses[i] - ref_loss) <= TOL[dtype] * max(1.0, abs(ref_loss))


def separated_setup(arch, n, seed, data_seed):
    net = Mo.build(arch)
    table, P = Mo.param_table(net)
    theta = synth.he_normal(table, P, seed)
    x, y = synth.batch(in_shape(arch), sum(n), data_seed, 1)
    if arch in ("mlp", "small_cnn"):
        # biases set on the whole batch: every worker's rows are separated too
        theta = separate_by_bias(net, theta, x, table, seed)
    else:
        theta = synth.separate_decisions(table, theta, seed)
    return net, table, theta, x, y


def exact_refs(net, table, theta, x, y, n, dtype, workers=None, log_margin=True):
    """The exact oracle's (loss, gradient, min ReLU margin, min pool margin)
    of every listed worker, and the oracle's floor at the path's precision."""
    refs = {}
    for i, (a, b) in enumerate(slices(n)):
        if workers is not None and i not in workers:
            continue
        if log_margin:
            log("  oracle worker %d (n=%d) ..." % (i, b - a))
        ctx = Mo.Ctx("exact")
        loss, g = Mo.worker_grad(net, theta.astype(np.float64), x[a:b], y[a:b], ctx=ctx)
        relu = min(m[1][0] for m in ctx.margins if m[0] == "relu" and m[1].size)
        pool = min((m[1][0] for m in ctx.margins if m[0] == "maxpool" and m[1].size),
                   default=1.0)
        floor = oracle_floor(net, theta, x[a:b], y[a:b], table, g, dtype)
        if log_margin:
            log("  oracle worker %d (n=%d): min relu margin %.1e, min pool margin %.1e"
                % (i, b - a, relu, pool))
        refs[i] = (loss, g, relu, pool, floor)
    return refs


def separated_problem(arch, dtype, n, seed):
    """Separated parameters and the first data seed whose ReLU decisions keep a
    margin of 1e-4 and whose max-pool decisions are unambiguous (fp32) in
    every worker."""
    for data_seed in range(seed, seed + 60):
        net, table, theta, x, y = separated_setup(arch, n, seed, data_seed)
        refs = exact_refs(net, table, theta, x, y, n, dtype, log_margin=False)
        if all(r[2] > 1e-4 and (r[3] > AMBIGUOUS["fp32"] or dtype == "bf16")
               for r in refs.values()):
            return net, table, theta, x, y, refs
    pytest.fail("no data seed with separated decisions in every worker")


# resnet18 bf16 [32, 1, 7, 24]: worker boundaries on the edges of the 512-row
# tiles of the 16x16, 8x8 and 4x4 maps (samples 32, 40, 64) and inside them
# (33), where the forward epilogue's batch-norm partials of consecutive
# workers meet
SEPARATED = [("resnet18", "fp32", [3, 1, 4]), ("resnet18", "bf16", [4, 2, 6, 1, 3]),
             ("resnet18", "bf16", [32, 1, 7, 24]),
             ("vgg16", "fp32", [2, 3]), ("vgg16", "bf16", [3, 5, 1]),
             ("resnet50", "fp32", [2, 1, 3]), ("resnet50", "bf16", [3, 5, 1, 2]),
             ("small_cnn", "bf16", [3, 4]), ("mlp", "bf16", [6, 17, 2])]


@pytest.mark.parametrize("arch,dtype,n", SEPARATED)
def test_workers_grad_separated(arch, dtype, n):
    """Separated decisions: every worker's gradient and loss against the exact
    oracle on its own rows, per tensor -- batch-norm statistics are the
    worker's own."""
    log("workers_grad separated %s %s n=%s" % (arch, dtype, n))
    net, table, theta, x, y, refs = separated_problem(arch, dtype, n, len(n))
    grads, losses = run_workers(arch, dtype, n, theta, x, y)
    for i, g in enumerate(grads):
        ref_loss, ref, _, _, floor = refs[i]
        assert np.all(np.isfinite(g))
        log("  worker %d (n=%d): loss %.6f vs %.6f" % (i, n[i], losses[i], ref_loss))
        check_pertensor(g, ref, table, TOL[dtype], floor=floor, what="worker %d vs exact" % i)
        assert abs(losses[i] - ref_loss) <= TOL[dtype] * max(1.0, abs(ref_loss))


@pytest.mark.parametrize("arch,dtype,n", [("resnet18", "fp32", [2, 5, 3]),
                                          ("vgg16", "bf16", [4, 1, 3]),
                                          ("resnet50", "bf16", [6, 2, 3]),
                                          ("resnet18", "bf16", [1, 1, 1, 1, 1, 1, 1, 761])])
def test_workers_grad_equals_separate_calls(arch, dtype, n):
    """One pass over all workers against one hs_worker_grad call per worker on
    the same rows (the two differ only in the order of fp32 sums, which can
    move a bf16 rounding), per tensor: the bar, or 3 x the oracle's floor at
    the path's precision for that worker where that exceeds it.  The last case
    puts several one-sample workers into one block of the 64-channel forward
    kernel, whose epilogue sums the batch-norm statistics per worker (N = 768:
    1536 half-image tiles over 256 blocks); its 761-sample worker fills the
    launch and is compared by its loss only (a float64 oracle pass over it,
    for its floor, takes minutes; the one-pass gradients of workers that size
    are compared with the oracle in the full-size tests)."""
    log("workers_grad vs worker_grad %s %s n=%s" % (arch, dtype, n))
    net = Mo.build(arch)
    table, P = Mo.param_table(net)
    theta = synth.separate_decisions(table, synth.he_normal(table, P, 3), 3)
    x, y = synth.batch((3, 32, 32), sum(n), 3, 1)
    ga, la = run_workers(arch, dtype, n, theta, x, y)
    gb, lb = run_workers(arch, dtype, n, theta, x, y, separate=True)
    small = [i for i in range(len(n)) if n[i] <= 64]
    refs = exact_refs(net, table, theta, x, y, n, dtype, workers=small, log_margin=False)
    for i in small:
        check_pertensor(ga[i], gb[i], table, TOL[dtype], floor=refs[i][4],
                        what="worker %d one pass vs separate" % i)
    for i in range(len(n)):
        assert np.all(np.isfinite(ga[i])) and np.all(np.isfinite(gb[i]))
    np.testing.assert_allclose(la, lb, rtol=TOL[dtype])


def test_workers_grad_deterministic():
    log("workers_grad determinism resnet18 bf16")
    n = [3, 6, 2]
    net = Mo.build("resnet18")
    table, P = Mo.param_table(net)
    theta = synth.he_normal(table, P, 5)
    x, y = synth.batch((3, 32, 32), sum(n), 5, 1)
    a = run_workers("resnet18", "bf16", n, theta, x, y)[0]
    b = run_workers("resnet18", "bf16", n, theta, x, y)[0]
    for ga, gb in zip(a, b):
        assert np.array_equal(ga, gb)


# ---------------------------------------------------------------------------
# the workload configurations at their own sizes (stored oracle values)
# ---------------------------------------------------------------------------
def load_golden(name):
    path = F.path(name)
    assert os.path.exists(path), "%s missing: python -m tests.golden.make_fullsize %s" % (path, name)
    return np.load(path)


def check_sampled(a, gold, prefix, table, idx, tol, what, floor_scale=1.0, ref=None):
    """Sampled per-tensor errors of a against the stored values `prefix`
    (or against `ref` sampled the same way, with the stored scales), bound
    max(tol, 3 x floor_scale x stored floor) on every tensor (the floor: the
    oracle's error at the path's precision over all of the tensor's
    entries); returns the worst (error, tensor)."""
    scales, vmax = gold[prefix + "_scale"], float(gold[prefix + "_vmax"])
    r = gold[prefix + "_ref"] if ref is None else np.concatenate([ref[ix] for ix in idx])
    errs = F.sampled_errors(a, r, idx, scales, vmax)
    fl = floor_scale * gold[prefix + "_floor"]
    bad, worst, within = [], (0.0, ""), 0
    for t, (row, e) in enumerate(zip(table, errs)):
        bound = max(tol, FLOOR_FACTOR * fl[t])
        within += e <= tol
        worst = max(worst, (e, row[0]))
        if not e <= bound:
            bad.append("%s %.3e > %.3e (floor %.3e)" % (row[0], e, bound, fl[t]))
    log("  %s: worst tensor %s %.3e; %d of %d tensors within %.0e (sampled, %d entries each)"
        % (what, worst[1], worst[0], within, len(errs), tol, F.SAMPLE))
    assert not bad, "%s: tensors beyond their bound: %s" % (what, "; ".join(bad[:8]))
    return worst


@pytest.mark.parametrize("name", [c[0] for c in F.FULL_SIZE])
def test_workers_grad_full_size(name):
    """A workload configuration at its own size, in one pass (the launch
    configuration the benchmark times), separated decisions: the compared
    workers against the exact oracle's stored values (tests/golden/
    make_fullsize.py), per tensor on sampled entries, from the one pass and
    from separate hs_worker_grad calls; every other worker's one-pass
    gradient against its separate call on all entries (fp32: the bar; bf16:
    two computations each within 3x the floor of exact differ by up to twice
    that, with the largest floor of the compared workers)."""
    _, arch, dtype, n, workers = F.CONFIGS[name]
    log("workers_grad full size %s n=%s" % (name, n))
    gold = load_golden(name)
    net, table, theta, x, y = F.setup(arch, n)
    np.testing.assert_allclose(F.fingerprint(theta, x, y), gold["fingerprint"], rtol=1e-9)
    assert list(gold["n"]) == list(n) and tuple(gold["workers"]) == tuple(workers)
    idx = F.sample_index(table)
    ga, la = run_workers(arch, dtype, n, theta, x, y)
    gb, lb = run_workers(arch, dtype, n, theta, x, y, separate=True)
    for i in range(len(n)):
        assert np.all(np.isfinite(ga[i])) and np.all(np.isfinite(gb[i])), "worker %d" % i
        check_padding(arch, ga[i])
    for i in workers:
        ref_loss = float(gold["w%d_loss" % i])
        log("  worker %d (n=%d): loss %.6f / %.6f vs %.6f, min relu margin %.1e"
            % (i, n[i], la[i], lb[i], ref_loss, float(gold["w%d_relu" % i])))
        check_sampled(ga[i], gold, "w%d" % i, table, idx, TOL[dtype], "worker %d one pass vs exact" % i)
        check_sampled(gb[i], gold, "w%d" % i, table, idx, TOL[dtype], "worker %d separate vs exact" % i)
        for loss in (la[i], lb[i]):
            assert abs(loss - ref_loss) <= TOL[dtype] * max(1.0, abs(ref_loss))
    fmax = np.max([gold["w%d_floor" % i] for i in workers], axis=0)
    for i in range(len(n)):
        if i in workers:
            continue
        errs = pertensor(ga[i], gb[i], table)
        bound = [max(TOL[dtype], FLOOR_FACTOR * 2.0 * f) if dtype == "bf16" else TOL[dtype]
                 for f in fmax]
        bad = ["%s %.3e > %.3e" % (nm, e, bd) for (nm, e, _), bd in zip(errs, bound) if not e <= bd]
        log("  worker %d (n=%d) one pass vs separate: worst %.3e" % (i, n[i], max(e for _, e, _ in errs)))
        assert not bad, "worker %d one pass vs separate: %s" % (i, "; ".join(bad[:8]))
        assert abs(la[i] - lb[i]) <= TOL[dtype] * max(1.0, abs(lb[i]))


def test_resnet18_fp32_full_size_step():
    """The ResNet-18 fp32 workload's step at its own size (N = 1024 over four
    workers 128/192/256/448, momentum 0.9, weight decay 5e-4, lr 0.1), all
    workers in one pass: the update theta' - theta and the momentum buffer
    after one step against the oracle's stored step (tests/golden/
    make_fullsize.py), per tensor on sampled entries."""
    require_gpu()
    from paper_2110_08941_amd.driver import Trainer
    log("full-size step resnet18_fp32 N=1024")
    gold = load_golden(F.STEP_NAME)
    wl = WORKLOADS["resnet18_fp32"]
    net = Mo.build(wl.arch)
    table, P = Mo.param_table(net)
    theta = synth.separate_decisions(table, synth.he_normal(table, P, F.STEP_SEED), F.STEP_SEED)
    tr = Trainer(wl, seed=F.STEP_SEED, clock="model", steps=1, theta0=theta, grouped=True)
    try:
        n = tr.part.partition()
        assert n == F.STEP_PARTITION
        x, y = tr.batch(0)
        np.testing.assert_allclose(F.fingerprint(theta, x.cpu().numpy(), y.cpu().numpy()),
                                   gold["fingerprint"], rtol=1e-9)
        tr.step()
        torch.cuda.synchronize()
        got = tr.theta.cpu().numpy().astype(np.float64)
        mom = tr.mom.cpu().numpy().astype(np.float64)
        losses = tr.losses.cpu().numpy()
    finally:
        tr.close()
    idx = F.sample_index(table)
    check_sampled(got - theta.astype(np.float64), gold, "d", table, idx, TOL["fp32"], "update")
    check_sampled(mom, gold, "buf", table, idx, TOL["fp32"], "momentum buffer")
    np.testing.assert_allclose(losses, gold["losses"], rtol=TOL["fp32"], atol=0)


@pytest.mark.parametrize("arch,dtype,n", [("resnet18", "bf16", [3, 5, 2]),
                                          ("resnet50", "bf16", [2, 3]),
                                          ("vgg16", "bf16", [4, 1, 3]),
                                          ("resnet18", "fp32", [2, 3])])
def test_single_stream_gives_identical_results(arch, dtype, n):
    """hs_workspace_set_streams(ws, 1) runs every launch on the caller's stream
    (the benchmark's per-kernel timings without overlap): the gradients and
    losses are bit-identical to the two-stream calls before and after it."""
    hs = require_gpu()
    log("single stream %s %s n=%s" % (arch, dtype, n))
    net = Mo.build(arch)
    table, P = Mo.param_table(net)
    theta = synth.separate_decisions(table, synth.he_normal(table, P, 9), 9)
    x, y = synth.batch((3, 32, 32), sum(n), 9, 1)
    m = hs.model_create(arch, dtype)
    try:
        th = torch.from_numpy(np.asarray(theta, dtype=np.float32)).cuda()
        tb = None
        if dtype == "bf16":
            tb = torch.empty(P, dtype=torch.int16, device="cuda")
            hs.params_to_bf16(th.data_ptr(), tb.data_ptr(), P)
        xd, yd = torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda()
        ws = hs.workspace_create(m, sum(n))
        out = []
        for streams in (2, 1, 1, 2):
            hs.workspace_set_streams(ws, streams)
            grads = [torch.full((P,), float("nan"), device="cuda") for _ in n]
            loss = torch.zeros(len(n), device="cuda")
            hs.workers_grad(m, ws, th.data_ptr(), tb.data_ptr() if tb is not None else 0,
                            xd.data_ptr(), yd.data_ptr(), n, [g.data_ptr() for g in grads],
                            loss.data_ptr(), 0)
            torch.cuda.synchronize()
            out.append(([g.cpu().numpy() for g in grads], loss.cpu().numpy()))
        with pytest.raises(hs.HSError):
            hs.workspace_set_streams(ws, 3)
        hs.workspace_destroy(ws)
    finally:
        hs.model_destroy(m)
    for k in range(1, 4):
        for a, b in zip(out[0][0], out[k][0]):
            assert np.array_equal(a, b)
        assert np.array_equal(out[0][1], out[k][1])


@pytest.mark.parametrize("arch,dtype,n", [("resnet18", "bf16", [3, 5, 2, 7]),
                                          ("resnet18", "fp32", [2, 3]),
                                          ("vgg16", "bf16", [4, 1, 3]),
                                          ("resnet50", "bf16", [2, 3, 1]),
                                          ("small_cnn", "fp32", [5, 9, 2]),
                                          ("mlp", "fp32", [64, 192]),
                                          ("mlp", "bf16", [7]),
                                          ("resnet18", "bf16", [52, 48, 49, 113, 119, 247, 177, 1243])])
def test_workers_grad_wavg_equals_weighted_average(arch, dtype, n):
    """hs_workers_grad_wavg (the partition weights applied in the per-worker
    reductions, one weighted gradient written) against hs_workers_grad
    followed by hs_weighted_average on the same inputs: bit-identical, as the
    header states (the same per-worker sums, combined in the same order and
    arithmetic).  The last case is the benchmark's N = 2048 launch."""
    hs = require_gpu()
    log("workers_grad_wavg %s %s n=%s" % (arch, dtype, n))
    net = Mo.build(arch)
    table, P = Mo.param_table(net)
    theta = synth.he_normal(table, P, 12)
    if arch not in ("mlp", "small_cnn"):
        theta = synth.separate_decisions(table, theta, 12)
    x, y = synth.batch(in_shape(arch), sum(n), 12, 1)
    m = hs.model_create(arch, dtype)
    try:
        th = torch.from_numpy(np.asarray(theta, dtype=np.float32)).cuda()
        tb = None
        if dtype == "bf16":
            tb = torch.empty(P, dtype=torch.int16, device="cuda")
            hs.params_to_bf16(th.data_ptr(), tb.data_ptr(), P)
        tbp = tb.data_ptr() if tb is not None else 0
        xd, yd = torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda()
        ws = hs.workspace_create(m, sum(n))
        grads = [torch.full((P,), float("nan"), device="cuda") for _ in n]
        la = torch.zeros(len(n), device="cuda")
        hs.workers_grad(m, ws, th.data_ptr(), tbp, xd.data_ptr(), yd.data_ptr(), n,
                        [g.data_ptr() for g in grads], la.data_ptr())
        avg = torch.full((P,), float("nan"), device="cuda")
        hs.weighted_average([g.data_ptr() for g in grads], n, P, avg.data_ptr())
        gbar = torch.full((P,), float("nan"), device="cuda")
        lb = torch.zeros(len(n), device="cuda")
        hs.workers_grad_wavg(m, ws, th.data_ptr(), tbp, xd.data_ptr(), yd.data_ptr(), n,
                             gbar.data_ptr(), lb.data_ptr())
        torch.cuda.synchronize()
        hs.workspace_destroy(ws)
        a, b = avg.cpu().numpy(), gbar.cpu().numpy()
    finally:
        hs.model_destroy(m)
    diff = np.flatnonzero(a.view(np.uint32) != b.view(np.uint32))
    log("  %d of %d entries differ" % (diff.size, P))
    assert diff.size == 0, "first differing entry %d: %r vs %r" % (diff[0], a[diff[0]], b[diff[0]])
    assert np.array_equal(la.cpu().numpy(), lb.cpu().numpy())
