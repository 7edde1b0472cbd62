"""The workload configurations at their own sizes, shared by the GPU tests and
the script that writes their stored oracle values (tests/golden/
make_fullsize.py, which calls only the oracle).

A float64 oracle pass over a worker of a thousand samples takes minutes, so
the oracle's values for these configurations are computed once, by that
script, and stored; the GPU tests compare sampled outputs with them: per
parameter tensor, SAMPLE seeded entries (every entry of smaller tensors),
with the tensor's largest exact magnitude (over all its entries) as the
denominator, as tests/gpu_util.pertensor does for whole tensors.  Inputs
(He-normal parameters, separated decisions, synthetic images) are drawn here
from their seeds on every machine; a fingerprint of them is stored with the
values and checked before any comparison.  A tensor's stored floor (the
oracle's own error at the path's precision) is its error over all entries,
not only the sampled ones: the sampled entries miss a tensor's worst ones,
and on the tensors where bf16 is most fragile that underestimates what a
valid bf16 computation is off by."""
import os

import numpy as np

from oracle import models as Mo
from paper_2110_08941_amd import synth

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
SAMPLE = 256
SEED = 11

# (name, arch, dtype, partition, workers compared with the oracle)
FULL_SIZE = [
    # ResNet-18 bf16, N = 2048 over 8 workers: a partition the benchmark's
    # drifting speeds reach
    ("resnet18_bf16_N2048", "resnet18", "bf16", [52, 48, 49, 113, 119, 247, 177, 1243],
     (0, 1, 2, 3, 4, 5, 6, 7)),
    # ResNet-18 fp32, N = 1024, speeds 1:1.5:2:3.5
    ("resnet18_fp32_N1024", "resnet18", "fp32", [128, 192, 256, 448], (0, 1, 2, 3)),
    # VGG-16 bf16, N = 4096, speeds 1:1:1:2:2:4:4:8: the smallest and the
    # largest worker
    ("vgg16_bf16_N4096", "vgg16", "bf16", [178, 178, 178, 356, 356, 713, 712, 1425], (0, 7)),
    # small CNN fp32, N = 512 at the partition of speeds 1:1:2:4
    ("small_cnn_fp32_N512", "small_cnn", "fp32", [64, 64, 128, 256], (0, 1, 2, 3)),
    # ResNet-50 bf16, N = 1024 over 8 workers: the two smallest workers
    ("resnet50_bf16_N1024", "resnet50", "bf16", [26, 24, 25, 56, 60, 123, 89, 621], (0, 1)),
]
CONFIGS = {c[0]: c for c in FULL_SIZE}

# rounding realizations behind a configuration's stored floors, where three
# (tests/gpu_util.REALIZATIONS) are too few: VGG-16's gradients behind its
# max-pool decisions have heavy-tailed bf16 errors (over 12 realizations of
# its smallest worker, the largest of the first 8 exceeds the largest of the
# first 3 by up to 1.9x, median 1.18x over the tensors)
REALIZATIONS_FULL = {"vgg16_bf16_N4096": (0, 1, 2, 3, 4, 5, 6, 7)}

# the ResNet-18 fp32 workload's step at its own size: partition, seed
STEP_NAME = "resnet18_fp32_step_N1024"
STEP_PARTITION = [128, 192, 256, 448]
STEP_SEED = 4


def in_shape(arch):
    return (784,) if arch == "mlp" else (3, 32, 32)


def slices(n):
    o = np.concatenate([[0], np.cumsum(n)]).astype(int)
    return [(int(o[i]), int(o[i + 1])) for i in range(len(n))]


def setup(arch, n, seed=SEED, data_seed=SEED):
    """(net, table, theta (float32), x, y) of a configuration: He-normal
    parameters with separated decisions (biases for BN-free networks, set on
    the whole batch), synthetic images."""
    from tests.gpu_util import separate_by_bias
    net = Mo.build(arch)
    table, P = Mo.param_table(net)
    theta = synth.he_normal(table, P, seed)
    x, y = synth.batch(in_shape(arch), sum(n), data_seed, 1)
    if arch in ("mlp", "small_cnn"):
        theta = separate_by_bias(net, theta, x, table, seed)
    else:
        theta = synth.separate_decisions(table, theta, seed)
    return net, table, theta, x, y


def fingerprint(*arrays):
    """Sum and sum of squares of each array, in float64."""
    out = []
    for a in arrays:
        a = np.asarray(a, dtype=np.float64)
        out += [float(a.sum()), float((a * a).sum())]
    return np.array(out)


def sample_index(table):
    """Per tensor, the flat indices of its sampled entries (all entries of a
    tensor with at most SAMPLE of them), drawn from a generator seeded with
    the tensor's position in the layout."""
    idx = []
    for t, row in enumerate(table):
        off, k = row[3], int(np.prod(row[2]))
        if k <= SAMPLE:
            idx.append(off + np.arange(k))
        else:
            rng = np.random.default_rng(1000 + t)
            idx.append(off + np.sort(rng.choice(k, SAMPLE, replace=False)))
    return idx


def tensor_scales(table, v):
    """max |v| per tensor over all its entries, and over the whole vector."""
    v = np.asarray(v, dtype=np.float64)
    scales = np.array([float(np.max(np.abs(v[r[3]:r[3] + int(np.prod(r[2]))])))
                       for r in table])
    return scales, float(np.max(np.abs(v)))


def full_errors(a, ref, table, scales, vmax):
    """Per tensor: max over all its entries of |a - ref| divided by the
    tensor's largest exact magnitude (at least ZERO_FLOOR of the whole
    vector's), ref the whole exact vector: the per-tensor error of
    tests/gpu_util.pertensor."""
    from tests.gpu_util import ZERO_FLOOR
    a = np.asarray(a, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    out = []
    for t, r in enumerate(table):
        off, k = r[3], int(np.prod(r[2]))
        d = float(np.max(np.abs(a[off:off + k] - ref[off:off + k])))
        den = max(float(scales[t]), ZERO_FLOOR * vmax)
        out.append(d / den if den > 0 else d)
    return out


def sampled_errors(a, ref_samples, idx, scales, vmax):
    """Per tensor: max over its sampled entries of |a - ref| divided by the
    tensor's largest exact magnitude (at least ZERO_FLOOR of the whole
    vector's, as pertensor)."""
    from tests.gpu_util import ZERO_FLOOR
    a = np.asarray(a, dtype=np.float64)
    out, o = [], 0
    for t, ix in enumerate(idx):
        r = np.asarray(ref_samples[o:o + len(ix)], dtype=np.float64)
        o += len(ix)
        den = max(float(scales[t]), ZERO_FLOOR * vmax)
        out.append(float(np.max(np.abs(a[ix] - r))) / den if den > 0 else
                   float(np.max(np.abs(a[ix] - r))))
    return out


def path(name):
    return os.path.join(GOLDEN, "fullsize_%s.npz" % name)
