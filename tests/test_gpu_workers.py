"""GPU parity of hs_workers_grad: all workers' gradients in one pass over the
layers (each layer launched once over the whole batch; batch-norm statistics,
losses and weight gradients per worker), checked worker by worker against the
oracle, and against separate hs_worker_grad calls.

Tolerances and the two decision regimes are those of test_gpu_worker.py:
normwise 1e-4 (fp32) / 2e-2 (bf16, oracle with bf16 storage); batch-norm
networks with separated decisions are compared directly, BN-free networks at
He init decision-aware.  Every case prints its name before it runs."""
import numpy as np
import pytest
import torch

from oracle import models as Mo
from paper_2110_08941_amd import synth
from tests.gpu_util import require_gpu, normwise, log
from tests.test_gpu_worker import decision_aware, check_padding, AMBIGUOUS

pytestmark = pytest.mark.gpu

TOL = {"fp32": 1e-4, "bf16": 2e-2}
STORAGE = {"fp32": "exact", "bf16": "bf16"}


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
           ("small_cnn", "fp32", [2, 1, 5, 3]), ("small_cnn", "bf16", [3, 4]),
           ("small_cnn", "fp32", [1] * 16),
           ("small_cnn", "fp32", [1, 2, 1, 3, 1, 1, 2, 1, 1, 1, 4, 1, 1, 2, 1, 3])]


@pytest.mark.parametrize("arch,dtype,n", HE_INIT)
def test_workers_grad_he_init(arch, dtype, n):
    """BN-free networks at He init: every worker's gradient and loss against
    the oracle on that worker's rows (decision-aware)."""
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
        err, namb, flips, ref_loss, _, _ = decision_aware(net, theta, x[a:b], y[a:b],
                                                         STORAGE[dtype], g)
        log("  worker %d (n=%d): normwise err %.3e (ambiguous %d, flipped %d) loss %.6f vs %.6f"
            % (i, b - a, err, namb, flips, losses[i], ref_loss))
        assert err <= TOL[dtype]
        assert abs(losses[i] - ref_loss) <= TOL[dtype] * max(1.0, abs(ref_loss))


SEPARATED = [("resnet18", "fp32", [3, 1, 4]), ("resnet18", "bf16", [4, 2, 6, 1, 3]),
             ("vgg16", "fp32", [2, 3]), ("vgg16", "bf16", [3, 5, 1]),
             ("resnet50", "fp32", [2, 1, 3]), ("resnet50", "bf16", [3, 5, 1, 2])]


def separated_problem(arch, dtype, n, seed):
    """Separated parameters and the first data seed whose ReLU decisions keep a
    margin of 1e-4 and whose max-pool decisions are unambiguous (fp32) in
    every worker."""
    net = Mo.build(arch)
    table, P = Mo.param_table(net)
    theta = synth.separate_decisions(table, synth.he_normal(table, P, seed), seed)
    for data_seed in range(seed, seed + 60):
        x, y = synth.batch((3, 32, 32), sum(n), data_seed, 1)
        refs, ok = [], True
        for a, b in slices(n):
            ctx = Mo.Ctx(STORAGE[dtype])
            loss, g = Mo.worker_grad(net, theta.astype(np.float64), x[a:b], y[a:b], ctx=ctx)
            relu = [m[1][0] for m in ctx.margins if m[0] == "relu" and m[1].size]
            pool = [m[1][0] for m in ctx.margins if m[0] == "maxpool" and m[1].size]
            ok = ok and min(relu) > 1e-4
            ok = ok and (min(pool, default=1.0) > AMBIGUOUS or dtype == "bf16")
            refs.append((loss, g))
        if ok:
            return net, theta, x, y, refs
    pytest.fail("no data seed with separated decisions in every worker")


@pytest.mark.parametrize("arch,dtype,n", SEPARATED)
def test_workers_grad_separated(arch, dtype, n):
    """Batch-norm networks (separated decisions): every worker's gradient and
    loss against the oracle on its own rows -- batch-norm statistics are the
    worker's own."""
    log("workers_grad separated %s %s n=%s" % (arch, dtype, n))
    net, theta, x, y, refs = separated_problem(arch, dtype, n, len(n))
    grads, losses = run_workers(arch, dtype, n, theta, x, y)
    for i, ((ref_loss, ref), g) in enumerate(zip(refs, grads)):
        assert np.all(np.isfinite(g))
        err = normwise(g, ref)
        log("  worker %d (n=%d): normwise err %.3e loss %.6f vs %.6f"
            % (i, n[i], err, losses[i], ref_loss))
        assert err <= TOL[dtype]
        assert abs(losses[i] - ref_loss) <= TOL[dtype] * max(1.0, abs(ref_loss))


@pytest.mark.parametrize("arch,dtype,n", [("resnet18", "fp32", [2, 5, 3]),
                                          ("vgg16", "bf16", [4, 1, 3]),
                                          ("resnet50", "bf16", [6, 2, 3]),
                                          ("resnet18", "bf16", [1, 1, 1, 1, 1, 1, 1, 761])])
def test_workers_grad_equals_separate_calls(arch, dtype, n):
    """One pass over all workers against one hs_worker_grad call per worker on
    the same rows (the two differ only in the order of fp32 sums).  The last
    case puts several one-sample workers into one block of the 64-channel
    forward kernel, whose epilogue sums the batch-norm statistics per worker
    (N = 768: 1536 half-image tiles over 256 blocks)."""
    log("workers_grad vs worker_grad %s %s n=%s" % (arch, dtype, n))
    net = Mo.build(arch)
    table, P = Mo.param_table(net)
    theta = synth.separate_decisions(table, synth.he_normal(table, P, 3), 3)
    x, y = synth.batch((3, 32, 32), sum(n), 3, 1)
    ga, la = run_workers(arch, dtype, n, theta, x, y)
    gb, lb = run_workers(arch, dtype, n, theta, x, y, separate=True)
    for i in range(len(n)):
        err = normwise(ga[i], gb[i])
        log("  worker %d: normwise difference %.3e" % (i, err))
        assert err <= TOL[dtype]
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


@pytest.mark.parametrize("arch,n", [
    ("resnet18", [52, 48, 49, 113, 119, 247, 177, 1243]),    # the benchmark, N = 2048
    ("resnet50", [26, 24, 25, 56, 60, 123, 89, 621])])        # N = 1024
def test_workers_grad_full_size_bench_configuration(arch, n):
    """The full-size launch configurations: bf16, 8 workers with a skewed
    partition, in one pass.  The two smallest workers are checked against the
    oracle (bf16 storage, separated decisions); every worker is checked
    against its own separate hs_worker_grad call."""
    log("workers_grad full size %s bf16 n=%s" % (arch, n))
    net = Mo.build(arch)
    table, P = Mo.param_table(net)
    theta = synth.separate_decisions(table, synth.he_normal(table, P, 11), 11)
    x, y = synth.batch((3, 32, 32), sum(n), 11, 1)
    ga, la = run_workers(arch, "bf16", n, theta, x, y)
    gb, lb = run_workers(arch, "bf16", n, theta, x, y, separate=True)
    for i in range(len(n)):
        assert np.all(np.isfinite(ga[i]))
        err = normwise(ga[i], gb[i])
        log("  worker %d (n=%d): vs separate call %.3e" % (i, n[i], err))
        assert err <= TOL["bf16"]
    np.testing.assert_allclose(la, lb, rtol=TOL["bf16"])
    sl = slices(n)
    for i in (1, 2):
        a, b = sl[i]
        ref_loss, ref = Mo.worker_grad(net, theta.astype(np.float64), x[a:b], y[a:b],
                                       storage="bf16")
        err = normwise(ga[i], ref)
        log("  worker %d (n=%d): vs oracle %.3e, loss %.6f vs %.6f"
            % (i, n[i], err, la[i], ref_loss))
        assert err <= TOL["bf16"]
        assert abs(la[i] - ref_loss) <= TOL["bf16"] * max(1.0, abs(ref_loss))


def test_workers_grad_rejects_bad_arguments():
    hs = require_gpu()
    m = hs.model_create("small_cnn", "fp32")
    try:
        P = hs.num_params(m)
        ws = hs.workspace_create(m, 8)
        th = torch.zeros(P, device="cuda")
        x = torch.zeros(8 * 3072, device="cuda")
        y = torch.zeros(8, dtype=torch.int32, device="cuda")
        g = [torch.zeros(P, device="cuda") for _ in range(17)]
        ptr = [t.data_ptr() for t in g]
        for n, gp in [([4, 5], ptr[:2]),            # sum above max_n
                      ([4, 0], ptr[:2]),            # empty worker
                      ([1] * 17, ptr)]:             # more than 16 workers
            with pytest.raises(hs.HSError):
                hs.workers_grad(m, ws, th.data_ptr(), 0, x.data_ptr(), y.data_ptr(), n, gp)
        hs.workspace_destroy(ws)
    finally:
        hs.model_destroy(m)


@pytest.mark.parametrize("arch,n", [("resnet18", [3, 5, 2]), ("resnet50", [2, 3]),
                                    ("vgg16", [4, 1, 3])])
def test_workers_grad_reused_workspace(arch, n):
    """A workspace's later calls (packed weights prepared on its second stream
    at the start of the call, from the current theta_bf16) give bit-identical
    gradients to a fresh workspace's first call (which packs as it goes), also
    after theta changed between the calls on the same stream."""
    hs = require_gpu()
    log("reused workspace %s bf16 n=%s" % (arch, n))
    net = Mo.build(arch)
    table, P = Mo.param_table(net)
    th1 = synth.separate_decisions(table, synth.he_normal(table, P, 7), 7)
    th2 = synth.separate_decisions(table, synth.he_normal(table, P, 8), 8)
    x, y = synth.batch((3, 32, 32), sum(n), 7, 1)
    m = hs.model_create(arch, "bf16")
    try:
        xd, yd = torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda()

        def call(ws, th):
            t = torch.from_numpy(np.asarray(th, dtype=np.float32)).cuda()
            tb = torch.empty(P, dtype=torch.int16, device="cuda")
            hs.params_to_bf16(t.data_ptr(), tb.data_ptr(), P)
            grads = [torch.full((P,), float("nan"), device="cuda") for _ in n]
            loss = torch.zeros(len(n), device="cuda")
            hs.workers_grad(m, ws, t.data_ptr(), tb.data_ptr(), xd.data_ptr(), yd.data_ptr(), n,
                            [g.data_ptr() for g in grads], loss.data_ptr(), 0)
            torch.cuda.synchronize()
            return [g.cpu().numpy() for g in grads], loss.cpu().numpy()

        ws = hs.workspace_create(m, sum(n))
        first = call(ws, th1)
        again = call(ws, th1)             # prepacked from the same theta
        changed = call(ws, th2)           # prepacked after theta changed
        hs.workspace_destroy(ws)
        fresh = hs.workspace_create(m, sum(n))
        ref2 = call(fresh, th2)
        hs.workspace_destroy(fresh)
    finally:
        hs.model_destroy(m)
    for a, b in zip(first[0], again[0]):
        assert np.array_equal(a, b)
    assert np.array_equal(first[1], again[1])
    for a, b in zip(changed[0], ref2[0]):
        assert np.array_equal(a, b)
    assert np.array_equal(changed[1], ref2[1])
    assert not np.array_equal(first[0][0], changed[0][0])
