"""The stored oracle values of the workload configurations at their own sizes
(tests/golden/fullsize_*.npz, written by tests/golden/make_fullsize.py) are
the committed oracle's: one worker of the small-CNN configuration is
recomputed here from the same seeds and compared with the stored entries;
every file's inputs fingerprint, partition and compared workers match the
configuration table, and its floors are whole-tensor errors (at least the
error on the sampled entries)."""
import os

import numpy as np
import pytest

from oracle import models as Mo
from tests import fullsize as F
from tests.gpu_util import REALIZATIONS


def test_small_cnn_worker_recomputed():
    name = "small_cnn_fp32_N512"
    _, arch, dtype, n, workers = F.CONFIGS[name]
    gold = np.load(F.path(name))
    net, table, theta, x, y = F.setup(arch, n)
    np.testing.assert_allclose(F.fingerprint(theta, x, y), gold["fingerprint"], rtol=1e-12)
    idx = F.sample_index(table)
    th = theta.astype(np.float64)
    a, b = F.slices(n)[0]
    loss, g = Mo.worker_grad(net, th, x[a:b], y[a:b])
    scales, vmax = F.tensor_scales(table, g)
    ref = np.concatenate([g[ix] for ix in idx])
    assert float(gold["w0_loss"]) == pytest.approx(loss, rel=1e-12)
    np.testing.assert_allclose(gold["w0_scale"], scales, rtol=1e-12)
    np.testing.assert_array_equal(gold["w0_ref"], ref.astype(np.float32))
    floors = []
    for k in REALIZATIONS[dtype]:
        _, gk = Mo.worker_grad(net, th, x[a:b], y[a:b], storage=dtype, grid=k)
        floors.append(F.full_errors(gk, g, table, scales, vmax))
    np.testing.assert_allclose(gold["w0_floor"], np.max(np.array(floors), axis=0), rtol=1e-9)


@pytest.mark.parametrize("name", [c[0] for c in F.FULL_SIZE])
def test_stored_files_match_configurations(name):
    _, arch, dtype, n, workers = F.CONFIGS[name]
    gold = np.load(F.path(name))
    assert list(gold["n"]) == list(n) and tuple(gold["workers"]) == tuple(workers)
    net, table, theta, x, y = F.setup(arch, n)
    np.testing.assert_allclose(F.fingerprint(theta, x, y), gold["fingerprint"], rtol=1e-12)
    idx = F.sample_index(table)
    sizes = [len(ix) for ix in idx]
    for i in workers:
        ref = np.split(gold["w%d_ref" % i].astype(np.float64), np.cumsum(sizes)[:-1])
        assert len(ref) == len(table) and ref[-1].size == sizes[-1]
        scale, floor = gold["w%d_scale" % i], gold["w%d_floor" % i]
        # a tensor's scale is its largest magnitude over all entries: at
        # least that of its sampled entries (float32-rounded)
        for t in range(len(table)):
            assert scale[t] >= np.max(np.abs(ref[t])) * (1 - 2.0 ** -23)
        assert np.all(np.isfinite(floor)) and np.all(floor >= 0)
        assert float(gold["w%d_vmax" % i]) == pytest.approx(float(np.max(scale)), rel=1e-12)
