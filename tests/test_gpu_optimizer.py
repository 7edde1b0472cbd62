"""GPU parity of the weighted average and the SGD update against the oracle
(Section 4.2 weighting; Section 1 / Section 5 update)."""
import numpy as np
import pytest
import torch

from oracle import step as S
from tests.gpu_util import require_gpu, normwise, rne_bf16_bits, dev, log

pytestmark = pytest.mark.gpu


def _case(P, M, seed):
    rng = np.random.default_rng(seed)
    g = [rng.standard_normal(P).astype(np.float32) for _ in range(M)]
    n = [int(v) for v in rng.integers(0, 300, size=M)]
    if sum(n) == 0:
        n[0] = 1
    theta = rng.standard_normal(P).astype(np.float32)
    mom = rng.standard_normal(P).astype(np.float32)
    return g, n, theta, mom


@pytest.mark.parametrize("P,M", [(1, 1), (5, 3), (64, 2), (1027, 8), (4096 * 37 + 3, 16),
                                 (203584, 2)])
def test_weighted_average(P, M):
    hs = require_gpu()
    log("weighted_average P=%d M=%d" % (P, M))
    g, n, _, _ = _case(P, M, seed=P + M)
    gd = [dev(v) for v in g]
    out = torch.empty(P, device="cuda")
    hs.weighted_average([t.data_ptr() for t in gd], n, P, out.data_ptr())
    torch.cuda.synchronize()
    ref = S.weighted_average(g, n)
    assert normwise(out.cpu().numpy(), ref) <= 1e-6


@pytest.mark.parametrize("P", [7, 1024, 99991])
@pytest.mark.parametrize("mu,wd,bf", [(0.0, 0.0, False), (0.9, 5e-4, False), (0.9, 5e-4, True),
                                      (0.0, 5e-4, True)])
def test_sgd_step(P, mu, wd, bf):
    hs = require_gpu()
    log("sgd_step P=%d mu=%g wd=%g bf16=%s" % (P, mu, wd, bf))
    g, _, theta, mom = _case(P, 1, seed=P)
    th_d, g_d = dev(theta), dev(g[0])
    mom_d = dev(mom) if mu != 0.0 else None
    tb = torch.zeros(P, dtype=torch.int16, device="cuda") if bf else None
    hs.sgd_step(th_d.data_ptr(), g_d.data_ptr(), mom_d.data_ptr() if mom_d is not None else 0, P,
                0.1, mu, wd, tb.data_ptr() if bf else 0)
    torch.cuda.synchronize()
    ref_t, ref_b = S.sgd_step(theta, g[0], mom if mu != 0.0 else None, 0.1, mu, wd)
    got = th_d.cpu().numpy()
    assert normwise(got - theta, ref_t - theta) <= 1e-5        # the update itself
    assert normwise(got, ref_t) <= 1e-6
    if mu != 0.0:
        assert normwise(mom_d.cpu().numpy(), ref_b) <= 1e-6
    if bf:
        assert np.array_equal(tb.cpu().numpy().view(np.uint16), rne_bf16_bits(got))


@pytest.mark.parametrize("P,M,mu,bf", [(4099, 4, 0.9, False), (64 * 1000, 8, 0.9, True),
                                       (17, 16, 0.0, False), (11174016, 8, 0.9, True)])
def test_wavg_sgd_fused(P, M, mu, bf):
    hs = require_gpu()
    log("wavg_sgd P=%d M=%d mu=%g bf16=%s" % (P, M, mu, bf))
    g, n, theta, mom = _case(P, M, seed=3 * P + M)
    gd = [dev(v) for v in g]
    th_d = dev(theta)
    mom_d = dev(mom) if mu != 0.0 else None
    tb = torch.zeros(P, dtype=torch.int16, device="cuda") if bf else None
    hs.wavg_sgd([t.data_ptr() for t in gd], n, th_d.data_ptr(),
                mom_d.data_ptr() if mom_d is not None else 0, P, 0.1, mu, 5e-4,
                tb.data_ptr() if bf else 0)
    torch.cuda.synchronize()
    gbar = S.weighted_average(g, n)
    ref_t, ref_b = S.sgd_step(theta, gbar, mom if mu != 0.0 else None, 0.1, mu, 5e-4)
    got = th_d.cpu().numpy()
    assert normwise(got - theta, ref_t - theta) <= 1e-5
    if mu != 0.0:
        assert normwise(mom_d.cpu().numpy(), ref_b) <= 1e-6
    if bf:
        assert np.array_equal(tb.cpu().numpy().view(np.uint16), rne_bf16_bits(got))


def test_wavg_sgd_standalone_size_sampled():
    """The standalone workload (8 fp32 buffers of 25M elements, partitions of
    the VGG-16 workload): sampled elements against the oracle's formula."""
    hs = require_gpu()
    from paper_2110_08941_amd.configs import STANDALONE_WAVG as W
    P, n = W["numel"], list(W["n"])
    log("wavg_sgd standalone P=%d" % P)
    gen = torch.Generator(device="cuda").manual_seed(5)
    gd = [torch.randn(P, device="cuda", generator=gen) for _ in range(len(n))]
    th = torch.randn(P, device="cuda", generator=gen)
    th0 = th.clone()
    hs.wavg_sgd([t.data_ptr() for t in gd], n, th.data_ptr(), 0, P, W["lr"], 0.0, 0.0)
    torch.cuda.synchronize()
    idx = torch.from_numpy(np.random.default_rng(1).integers(0, P, size=200000)).cuda()
    gs = [t[idx].cpu().numpy() for t in gd]
    ref, _ = S.sgd_step(th0[idx].cpu().numpy(), S.weighted_average(gs, n), None, W["lr"], 0.0, 0.0)
    got = th[idx].cpu().numpy()
    base = th0[idx].cpu().numpy()
    assert normwise(got - base, ref - base) <= 1e-5


def test_deterministic():
    hs = require_gpu()
    g, n, theta, mom = _case(300001, 8, seed=9)
    outs = []
    for _ in range(2):
        gd = [dev(v) for v in g]
        th = dev(theta)
        mo = dev(mom)
        hs.wavg_sgd([t.data_ptr() for t in gd], n, th.data_ptr(), mo.data_ptr(), 300001, 0.1, 0.9,
                    5e-4, 0)
        torch.cuda.synchronize()
        outs.append((th.cpu().numpy(), mo.cpu().numpy()))
    assert np.array_equal(outs[0][0], outs[1][0]) and np.array_equal(outs[0][1], outs[1][1])
