"""The allocation-free variant of the one-pass worker gradients
(hs_workers_grad_static: its scratch is the library's static device buffer)
against hs_workers_grad with a workspace, through the C ABI: two calls in a
row, the second with a smaller input, each against a workspace call on the
same rows; every worker's gradient per tensor within the parity bar (1e-4
fp32, 2e-2 bf16 -- the two split the weight-gradient sums differently), the
losses too; a request beyond the buffer is refused before any launch."""
import numpy as np
import pytest
import torch

from oracle import models as Mo
from paper_2110_08941_amd import synth
from tests.gpu_util import require_gpu, log, TOL, check_pertensor

pytestmark = pytest.mark.gpu


def in_shape(arch):
    return (784,) if arch == "mlp" else (3, 32, 32)


def grads(hs, m, arch, dtype, n, theta, x, y, static):
    P = hs.num_params(m)
    th = torch.from_numpy(np.asarray(theta, dtype=np.float32)).cuda()
    tb = None
    if dtype == "bf16":
        tb = torch.empty(P, dtype=torch.int16, device="cuda")
        hs.params_to_bf16(th.data_ptr(), tb.data_ptr(), P)
    xd, yd = torch.from_numpy(x).cuda(), torch.from_numpy(y).cuda()
    g = [torch.full((P,), float("nan"), device="cuda") for _ in n]
    loss = torch.full((len(n),), float("nan"), device="cuda")
    tbp = tb.data_ptr() if tb is not None else 0
    if static:
        hs.workers_grad_static(m, th.data_ptr(), tbp, xd.data_ptr(), yd.data_ptr(), n,
                               [t.data_ptr() for t in g], loss.data_ptr())
    else:
        ws = hs.workspace_create(m, sum(n))
        hs.workers_grad(m, ws, th.data_ptr(), tbp, xd.data_ptr(), yd.data_ptr(), n,
                        [t.data_ptr() for t in g], loss.data_ptr())
        torch.cuda.synchronize()
        hs.workspace_destroy(ws)
    torch.cuda.synchronize()
    return [t.cpu().numpy() for t in g], loss.cpu().numpy()


CASES = [("mlp", "fp32", [64, 192], [5, 11]),
         ("small_cnn", "fp32", [6, 20, 9], [3, 2]),
         ("small_cnn", "bf16", [40, 50, 30], [7]),
         ("resnet18", "bf16", [1, 3, 1], [2, 1]),
         ("vgg16", "bf16", [2, 3], [1, 1, 1])]


@pytest.mark.parametrize("arch,dtype,n1,n2", CASES)
def test_static_variant_matches_workspace_call(arch, dtype, n1, n2):
    hs = require_gpu()
    log("workers_grad_static %s %s n=%s then n=%s" % (arch, dtype, n1, n2))
    net = Mo.build(arch)
    table, P = Mo.param_table(net)
    m = hs.model_create(arch, dtype)
    try:
        for call, n in enumerate((n1, n2)):
            theta = synth.he_normal(table, P, 40 + call)
            if arch not in ("mlp", "small_cnn"):
                theta = synth.separate_decisions(table, theta, 40 + call)
            x, y = synth.batch(in_shape(arch), sum(n), 40 + call, 1)
            gs, ls = grads(hs, m, arch, dtype, n, theta, x, y, static=True)
            gw, lw = grads(hs, m, arch, dtype, n, theta, x, y, static=False)
            for i in range(len(n)):
                assert np.all(np.isfinite(gs[i])), "worker %d: not fully written" % i
                check_pertensor(gs[i], gw[i], table, TOL[dtype],
                                what="call %d worker %d static vs workspace" % (call, i))
            np.testing.assert_allclose(ls, lw, rtol=TOL[dtype])
    finally:
        hs.model_destroy(m)


def test_static_variant_rejects_sizes_beyond_its_buffer():
    hs = require_gpu()
    m = hs.model_create("resnet18", "bf16")
    try:
        P = hs.num_params(m)
        big = 64
        assert hs.workers_grad_static_bytes(m, big) > 128 << 20
        th = torch.zeros(P, device="cuda")
        tb = torch.zeros(P, dtype=torch.int16, device="cuda")
        x = torch.zeros(big * 3072, device="cuda")
        y = torch.zeros(big, dtype=torch.int32, device="cuda")
        g = torch.full((P,), 7.0, device="cuda")
        with pytest.raises(hs.HSError) as e:
            hs.workers_grad_static(m, th.data_ptr(), tb.data_ptr(), x.data_ptr(), y.data_ptr(),
                                   [big], [g.data_ptr()])
        assert e.value.status == hs.HS_ERR_INVALID and "static buffer" in str(e.value)
        torch.cuda.synchronize()
        assert torch.all(g == 7.0)          # nothing was launched
    finally:
        hs.model_destroy(m)
