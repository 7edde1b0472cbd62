"""GPU parity of the worker gradient (hs_worker_grad) against the oracle.

Error measure: per parameter tensor, max |a - b| / max |b| (every tensor of the
layout, the worst one named on failure).  The reference is the exact float64
oracle (storage "exact", the definition of Eq. (1)) in every test; the bar is
1e-4 (fp32) / 2e-2 (bf16) on every tensor where the arithmetic of that
precision permits it.  In the deep batch-norm networks it does not everywhere:
rounding alone -- the oracle's own arithmetic in fp32 or bf16 (contraction
operands and every tensor between layers rounded, sums exact) -- moves
batch-norm shift gradients that are residues of cancelling sums by more than
the bar (a few 1e-4 in fp32, up to tens of percent in bf16), and bf16 more
than that on most tensors of ResNet-18 and VGG-16 (rounding alone the
contraction operands already does, which the bf16 path does by definition).
On a tensor where that floor exceeds the bar the bound is 3 x the floor; every
test logs how many tensors meet the bar outright.

Decisions.  A ReLU whose input is within the arithmetic's rounding error of
zero may go either way; both outcomes are correct, and in deep batch-norm
networks one such flip moves gradient entries by percents.  Regimes:
  * He init (the workloads' distribution), BN-free networks: the oracle lists
    every ReLU decision within a margin of zero (1e-6 relative in fp32, 5e-3
    in bf16) and computes the gradient change of flipping each; the GPU result
    must equal the oracle's for SOME choice of those flips (least squares,
    rounded to 0/1), within the tolerance;
  * separated: batch-norm parameters (synth.separate_decisions), or for
    BN-free networks biases (separate_by_bias), that keep every ReLU input far
    from zero; the comparison is direct.
Every case prints its name before it runs."""
import numpy as np
import pytest
import torch

from oracle import models as Mo
from paper_2110_08941_amd import synth
from tests.gpu_util import (require_gpu, normwise, dev, log, TOL, pertensor, check_pertensor,
                            separate_by_bias, oracle_floor)

pytestmark = pytest.mark.gpu

AMBIGUOUS = {"fp32": 1e-6, "bf16": 5e-3}


def in_shape(arch):
    return (784,) if arch == "mlp" else (3, 32, 32)


def run_worker(arch, dtype, n, seed=0, theta=None, data_seed=None):
    """GPU gradient of one worker on n synthetic samples; returns
    (theta, x, y, g_gpu, loss_gpu)."""
    hs = require_gpu()
    m = hs.model_create(arch, dtype)
    try:
        table = hs.param_table(m)
        P = hs.num_params(m)
        if theta is None:
            theta = synth.he_normal(table, P, seed)
        x, y = synth.batch(in_shape(arch), n, seed if data_seed is None else data_seed, 1)
        th_d = dev(theta)
        tb = None
        if dtype == "bf16":
            tb = torch.empty(P, dtype=torch.int16, device="cuda")
            hs.params_to_bf16(th_d.data_ptr(), tb.data_ptr(), P)
        x_d, y_d = dev(x), dev(y)
        g_d = torch.full((P,), float("nan"), device="cuda")     # must be fully overwritten
        loss_d = torch.zeros(1, device="cuda")
        ws = hs.workspace_create(m, n)
        hs.worker_grad(m, ws, th_d.data_ptr(), tb.data_ptr() if tb is not None else 0,
                       x_d.data_ptr(), y_d.data_ptr(), n, g_d.data_ptr(), loss_d.data_ptr(), 0)
        torch.cuda.synchronize()
        hs.workspace_destroy(ws)
        return theta, x, y, g_d.cpu().numpy(), float(loss_d.cpu()[0])
    finally:
        hs.model_destroy(m)


def decision_aware(net, theta, x, y, g_gpu, capture):
    """The exact oracle's gradient with the outcomes of its ambiguous ReLU
    decisions (margin below `capture`) chosen to fit g_gpu: least squares over
    the flip directions, rounded to 0/1.  Returns (reference, n_ambiguous,
    flips, loss)."""
    th = np.asarray(theta, dtype=np.float64)
    ctx = Mo.Ctx("exact", capture=capture)
    loss, g0 = Mo.worker_grad(net, th, x, y, ctx=ctx)
    amb = [(c, i) for c, i, _ in ctx.ambiguous]
    if not amb:
        return g0, 0, 0, loss
    D = np.stack([Mo.worker_grad(net, th, x, y, ctx=Mo.Ctx("exact", toggles={a}))[1] - g0
                  for a in amb], axis=1)
    s = np.linalg.lstsq(D, np.asarray(g_gpu, dtype=np.float64) - g0, rcond=None)[0]
    s = np.clip(np.round(s), 0.0, 1.0)
    return g0 + D @ s, len(amb), int(s.sum()), loss


def check_padding(arch, g):
    net = Mo.build(arch)
    table, P = Mo.param_table(net)
    used = np.zeros(P, dtype=bool)
    for name, kind, shape, off in table:
        used[off:off + int(np.prod(shape))] = True
    assert np.all(g[~used] == 0.0)


HE_INIT = [("mlp", "fp32", 1), ("mlp", "fp32", 7), ("mlp", "fp32", 64),
           ("small_cnn", "fp32", 1), ("small_cnn", "fp32", 5), ("small_cnn", "fp32", 19),
           ("mlp", "bf16", 9), ("mlp", "bf16", 64)]


@pytest.mark.parametrize("arch,dtype,n", HE_INIT)
def test_worker_grad_he_init(arch, dtype, n):
    """BN-free networks at the workloads' He init against the exact oracle,
    decision-aware, 1e-4 (fp32) / 2e-2 (bf16) on every tensor."""
    log("worker_grad he-init %s %s n=%d" % (arch, dtype, n))
    theta, x, y, g, loss = run_worker(arch, dtype, n, seed=n)
    assert np.all(np.isfinite(g)), "gradient has non-finite entries"
    check_padding(arch, g)
    net = Mo.build(arch)
    table, _ = Mo.param_table(net)
    ref, namb, flips, ref_loss = decision_aware(net, theta, x, y, g, AMBIGUOUS[dtype])
    log("  ambiguous ReLU %d, flipped %d, loss %.6f vs %.6f" % (namb, flips, loss, ref_loss))
    check_pertensor(g, ref, table, TOL[dtype], what="gradient vs exact")
    assert abs(loss - ref_loss) <= TOL[dtype] * max(1.0, abs(ref_loss))


def separated_theta(arch, n, seed, dtype, data_seed):
    """Parameters of the separated regime for a data batch."""
    net = Mo.build(arch)
    table, P = Mo.param_table(net)
    theta = synth.he_normal(table, P, seed)
    x, y = synth.batch(in_shape(arch), n, data_seed, 1)
    if arch in ("mlp", "small_cnn"):
        theta = separate_by_bias(net, theta, x, table, seed)
    else:
        theta = synth.separate_decisions(table, theta, seed)
    return net, table, theta, x, y


def separated_problem(arch, dtype, n, seed):
    """The first data seed whose ReLU margins exceed 1e-4 and, in fp32, whose
    max-pool margins exceed 1e-6 in the exact oracle; returns the problem and
    the oracle's exact gradient and loss."""
    for data_seed in range(seed, seed + 60):
        net, table, theta, x, y = separated_theta(arch, n, seed, dtype, data_seed)
        ctx = Mo.Ctx("exact")
        ref_loss, ref = Mo.worker_grad(net, theta.astype(np.float64), x, y, ctx=ctx)
        relu = [m[1][0] for m in ctx.margins if m[0] == "relu" and m[1].size]
        pool = [m[1][0] for m in ctx.margins if m[0] == "maxpool" and m[1].size]
        if min(relu) > 1e-4 and (min(pool, default=1.0) > AMBIGUOUS["fp32"] or dtype == "bf16"):
            return net, table, theta, x, y, data_seed, ref_loss, ref, min(relu)
    pytest.fail("no data seed with separated ReLU and unambiguous max-pool decisions")


SEPARATED = [("resnet18", "fp32", 4), ("resnet18", "fp32", 13),
             ("vgg16", "fp32", 4), ("vgg16", "fp32", 6),
             ("resnet50", "fp32", 3), ("resnet50", "fp32", 10),
             ("small_cnn", "bf16", 3), ("small_cnn", "bf16", 11),
             ("mlp", "bf16", 33),
             ("resnet18", "bf16", 4), ("resnet18", "bf16", 16),
             ("vgg16", "bf16", 4), ("vgg16", "bf16", 12),
             ("resnet50", "bf16", 4), ("resnet50", "bf16", 9)]


@pytest.mark.parametrize("arch,dtype,n", SEPARATED)
def test_worker_grad_separated(arch, dtype, n):
    """Every ReLU decision far from zero: the GPU gradient against the exact
    oracle on every tensor (the bar, or 3 x the oracle's floor at the path's
    precision where that exceeds it)."""
    log("worker_grad separated %s %s n=%d" % (arch, dtype, n))
    net, table, theta, x, y, data_seed, ref_loss, ref, margin = separated_problem(arch, dtype, n, n)
    _, _, _, g, loss = run_worker(arch, dtype, n, theta=theta, data_seed=data_seed)
    assert np.all(np.isfinite(g))
    check_padding(arch, g)
    floor = oracle_floor(net, theta, x, y, table, ref, dtype)
    log("  min relu margin %.1e, data seed %d, loss %.6f vs %.6f" % (margin, data_seed, loss, ref_loss))
    check_pertensor(g, ref, table, TOL[dtype], floor=floor, what="gradient vs exact")
    assert abs(loss - ref_loss) <= TOL[dtype] * max(1.0, abs(ref_loss))


@pytest.mark.parametrize("arch,dtype,n", [("small_cnn", "fp32", 37), ("resnet18", "bf16", 19),
                                          ("vgg16", "fp32", 5)])
def test_worker_grad_deterministic(arch, dtype, n):
    log("determinism %s %s n=%d" % (arch, dtype, n))
    a = run_worker(arch, dtype, n, seed=2)[3]
    b = run_worker(arch, dtype, n, seed=2)[3]
    assert np.array_equal(a, b)
