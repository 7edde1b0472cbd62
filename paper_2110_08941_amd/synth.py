"""Seeded synthetic inputs (no arithmetic of the method lives here).

The paper trains on CIFAR10 (Section 5); that dataset is not available, so the
workloads use synthetic data of the same shape: 3x32x32 images with pixels
drawn from N(0, 1) and labels uniform over 10 classes (a flat 784-vector for
the MLP workload).  Parameters are He-normal (std = sqrt(2 / fan_in)), biases
and batch-norm beta zero, batch-norm gamma one.

Both the GPU library and the CPU oracle receive the arrays made here; neither
draws random numbers of its own.
"""
import numpy as np

_TAG_BATCH, _TAG_PARAM, _TAG_SPEED = 11, 12, 13


def _rng(*key):
    return np.random.default_rng(np.random.SeedSequence([int(k) for k in key]))


def batch(in_shape, total, seed, step, classes=10):
    """x float32 [total, *in_shape] ~ N(0, 1); y int32 [total] ~ U{0..classes-1}.
    One fresh batch per (seed, step)."""
    g = _rng(seed, _TAG_BATCH, step)
    x = g.standard_normal((total,) + tuple(in_shape), dtype=np.float32)
    y = g.integers(0, classes, size=total, dtype=np.int32)
    return x, y


def fan_in(kind, shape):
    if kind == "conv_w":          # [c_out, kh, kw, c_in]
        return shape[1] * shape[2] * shape[3]
    if kind == "lin_w":           # [out, in]
        return shape[1]
    return None


def he_normal(table, total, seed):
    """Flat float32 parameter vector of length `total` for a tensor table of
    (name, kind, shape, offset) rows; padding gaps stay zero."""
    theta = np.zeros(total, dtype=np.float32)
    g = _rng(seed, _TAG_PARAM)
    for name, kind, shape, off in table:
        numel = int(np.prod(shape))
        if kind in ("conv_w", "lin_w"):
            std = np.sqrt(2.0 / fan_in(kind, shape))
            theta[off:off + numel] = (g.standard_normal(numel) * std).astype(np.float32)
        elif kind == "bn_gamma":
            theta[off:off + numel] = 1.0
        else:                      # bias, bn_beta
            theta[off:off + numel] = 0.0
    return theta


def separate_decisions(table, theta, seed, gamma=0.5, shift=3.0):
    """Batch-norm parameters that keep every ReLU decision far from its
    threshold (for exact comparisons of deep ReLU/BN networks): gamma = 0.5
    and beta = +shift on every channel of a batch-norm that feeds a residual
    sum (in a residual block "layerS.B", the projection's batch-norm and the
    highest-numbered "bnK" of the block: bn2 of a basic block, bn3 of a
    bottleneck) and on a batch-norm named "bn2" outside residual blocks
    (VGG-16's second), and beta = +shift or -shift on a random half of the
    channels of every other batch-norm.  With |xhat| below shift / gamma, every
    pre-activation is then >= shift - gamma |xhat| away from zero.  Returns a
    modified copy of theta."""
    th = np.array(theta, dtype=np.float32, copy=True)
    g = _rng(seed, 19)
    last_bn = {}
    for name, kind, shape, off in table:
        block, _, leaf = name.rpartition(".")[0].rpartition(".")
        if kind == "bn_beta" and name.startswith("layer") and leaf.startswith("bn"):
            last_bn[block] = max(last_bn.get(block, 0), int(leaf[2:]))
    for name, kind, shape, off in table:
        numel = int(np.prod(shape))
        block, _, leaf = name.rpartition(".")[0].rpartition(".")
        if name.startswith("layer"):
            residual = "proj_bn" in name or (leaf.startswith("bn") and
                                             int(leaf[2:]) == last_bn.get(block))
        else:
            residual = name.split(".")[0] == "bn2"
        if kind == "bn_gamma":
            th[off:off + numel] = gamma
        elif kind == "bn_beta":
            if residual:
                th[off:off + numel] = shift
            else:
                sign = np.where(g.random(numel) < 0.5, -1.0, 1.0)
                th[off:off + numel] = (sign * shift).astype(np.float32)
    return th


def speed_schedule(base, steps, seed, drift_sigma=0.0):
    """Per-step worker speeds s_m(t), t = 0..steps-1, as float64 [steps, M].

    Without drift every step uses `base`.  With drift the speeds follow a
    multiplicative random walk s_m(t) = s_m(t-1) * exp(sigma * z), z ~ N(0, 1),
    applied before step t is timed (so step 0 already carries one draw)."""
    base = np.asarray(base, dtype=np.float64)
    out = np.empty((steps, base.size), dtype=np.float64)
    s = base.copy()
    for t in range(steps):
        if drift_sigma > 0.0:
            z = _rng(seed, _TAG_SPEED, t).standard_normal(base.size)
            s = s * np.exp(drift_sigma * z)
        out[t] = s
    return out


def random_buffers(count, numel, seed, dtype=np.float32):
    """`count` arrays of `numel` N(0, 1) values (standalone reduction bench)."""
    g = _rng(seed, 17)
    return [g.standard_normal(numel, dtype=np.float32).astype(dtype) for _ in range(count)]
