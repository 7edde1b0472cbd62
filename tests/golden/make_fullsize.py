"""Writes the oracle's values for the workload configurations at their own
sizes (tests/fullsize.py) into tests/golden/fullsize_<name>.npz.  Calls only
the oracle and the seeded input generators; runs on the CPU (a float64 pass
over a thousand ResNet-18 samples takes minutes, the whole set about two
hours on eight cores).

    python -m tests.golden.make_fullsize [name ...]      (default: all)

Per compared worker i of a configuration (Eq. (1): the mean gradient over
the worker's own partition):
  w<i>_loss        the worker's mean loss
  w<i>_scale       per tensor, max |g| over all its entries
  w<i>_vmax        max |g| over the whole vector
  w<i>_ref         g at the sampled entries (fullsize.sample_index), float32
  w<i>_floor       per tensor, the error (over all its entries) of the
                   oracle's own arithmetic at the path's precision (Ctx
                   modes "fp32" / "bf16"), the largest over the precision's
                   rounding realizations (fullsize.REALIZATIONS_FULL where
                   a configuration needs more than tests.gpu_util's)
  w<i>_relu        the smallest ReLU margin of the exact pass
and the configuration's partition, compared workers and input fingerprint.
The step file holds the same for the update theta' - theta ("d_") and the
momentum buffer ("buf_") of one step of the ResNet-18 fp32 workload
(Section 4.2 average, momentum SGD), the floors from the oracle's fp32 step
with theta' stored in fp32."""
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from oracle import models as Mo                       # noqa: E402
from oracle import step as S                          # noqa: E402
from paper_2110_08941_amd import synth                # noqa: E402
from paper_2110_08941_amd.configs import WORKLOADS    # noqa: E402
from tests import fullsize as F                       # noqa: E402
from tests.gpu_util import REALIZATIONS               # noqa: E402


def say(msg):
    print("[%s] %s" % (time.strftime("%H:%M:%S"), msg), flush=True)


def summarize(table, idx, v):
    scales, vmax = F.tensor_scales(table, v)
    ref = np.concatenate([np.asarray(v, dtype=np.float64)[ix] for ix in idx])
    return scales, vmax, ref


def make_config(name):
    _, arch, dtype, n, workers = F.CONFIGS[name]
    net, table, theta, x, y = F.setup(arch, n)
    idx = F.sample_index(table)
    th = theta.astype(np.float64)
    out = {"n": np.array(n), "workers": np.array(workers),
           "fingerprint": F.fingerprint(theta, x, y)}
    for i in workers:
        a, b = F.slices(n)[i]
        say("%s worker %d (n=%d): exact" % (name, i, b - a))
        ctx = Mo.Ctx("exact")
        loss, g = Mo.worker_grad(net, th, x[a:b], y[a:b], ctx=ctx)
        relu = min(m[1][0] for m in ctx.margins if m[0] == "relu" and m[1].size)
        scales, vmax, ref = summarize(table, idx, g)
        floors = []
        for k in F.REALIZATIONS_FULL.get(name, REALIZATIONS[dtype]):
            say("%s worker %d: %s realization %d" % (name, i, dtype, k))
            _, gk = Mo.worker_grad(net, th, x[a:b], y[a:b], storage=dtype, grid=k)
            floors.append(F.full_errors(gk, g, table, scales, vmax))
        out["w%d_loss" % i] = np.array(loss)
        out["w%d_scale" % i] = scales
        out["w%d_vmax" % i] = np.array(vmax)
        out["w%d_ref" % i] = ref.astype(np.float32)
        out["w%d_floor" % i] = np.max(np.array(floors), axis=0)
        out["w%d_relu" % i] = np.array(relu)
    return out


def make_step():
    wl = WORKLOADS["resnet18_fp32"]
    net = Mo.build(wl.arch)
    table, P = Mo.param_table(net)
    theta = synth.separate_decisions(table, synth.he_normal(table, P, F.STEP_SEED), F.STEP_SEED)
    x, y = synth.batch(wl.in_shape, wl.total, F.STEP_SEED, 0)
    n = F.STEP_PARTITION
    idx = F.sample_index(table)
    th = theta.astype(np.float64)

    def worker(mode):
        def grad(t, xm, ym):
            say("step worker n=%d (%s)" % (len(ym), mode))
            return Mo.worker_grad(net, t, xm, ym, storage=mode)
        return grad

    ex = S.step(worker("exact"), th, None, x, y, n, wl.lr, wl.mu, wl.wd)
    lo = S.step(worker("fp32"), th, None, x, y, n, wl.lr, wl.mu, wl.wd)
    out = {"n": np.array(n), "fingerprint": F.fingerprint(theta, x, y)}
    d_ref = ex["theta"] - th
    d_low = lo["theta"].astype(np.float32).astype(np.float64) - th   # fp32 master weights
    for key, ref_v, low_v in (("d", d_ref, d_low), ("buf", ex["buf"], lo["buf"])):
        scales, vmax, ref = summarize(table, idx, ref_v)
        out[key + "_scale"] = scales
        out[key + "_vmax"] = np.array(vmax)
        out[key + "_ref"] = ref.astype(np.float32)
        out[key + "_floor"] = np.array(F.full_errors(low_v, ref_v, table, scales, vmax))
    out["losses"] = np.array(ex["losses"])
    return out


def main(names):
    os.makedirs(F.GOLDEN, exist_ok=True)
    for name in names:
        t0 = time.time()
        out = make_step() if name == F.STEP_NAME else make_config(name)
        np.savez_compressed(F.path(name), **out)
        say("%s written (%.0f s)" % (name, time.time() - t0))


if __name__ == "__main__":
    main(sys.argv[1:] or [F.STEP_NAME] + [c[0] for c in F.FULL_SIZE])
