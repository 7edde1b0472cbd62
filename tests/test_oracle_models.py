"""Pins of the oracle's per-worker gradients (CPU only).

* central finite differences on small networks of every layer type;
* an independent implementation: the same networks written with
  torch.nn.functional in float64, differentiated by autograd;
* the invariant of Eq. (1) with the partition-size weights of Section 4.2:
  for networks without batch-norm, the weighted average of the per-partition
  mean gradients equals the full-batch mean gradient, for any partition;
* the parameter counts of the four networks.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import models as Mo
from oracle import step as S

TINY = {
    "mlp": (dict(in_dim=8, hidden=6, classes=3), (8,), 5),
    "small_cnn": (dict(in_ch=3, widths=(2, 3, 4), classes=3), (3, 6, 6), 4),
    "resnet18": (dict(in_ch=3, widths=(3, 4), blocks=(1, 2), classes=3), (3, 8, 8), 3),
    # bottlenecks with a stride-1 projection, an identity shortcut and a
    # stride-2 projection
    "resnet50": (dict(in_ch=3, widths=(2, 3), blocks=(2, 1), expansion=2, classes=3), (3, 8, 8), 3),
    "vgg16": (dict(in_ch=3, cfg=(3, "M", 4, 4, "M"), fc_hidden=5, classes=3), (3, 4, 4), 4),
}


def rand_problem(arch, kw, in_shape, n, seed):
    net = Mo.build(arch, **kw)
    table, total = Mo.param_table(net)
    rng = np.random.default_rng(seed)
    theta = np.zeros(total)
    for name, kind, shape, off in table:
        k = int(np.prod(shape))
        theta[off:off + k] = rng.standard_normal(k) * (0.7 if kind in ("conv_w", "lin_w") else 0.3)
        if kind == "bn_gamma":
            theta[off:off + k] += 1.0
    x = rng.standard_normal((n,) + in_shape)
    y = rng.integers(0, kw.get("classes", 10), size=n)
    return net, table, total, theta, x, y


@pytest.mark.parametrize("arch", sorted(TINY))
def test_finite_differences(arch):
    kw, in_shape, n = TINY[arch]
    net, table, total, theta, x, y = rand_problem(arch, kw, in_shape, n, seed=11)
    loss, g = Mo.worker_grad(net, theta, x, y)
    rng = np.random.default_rng(1)
    coords = []
    for name, kind, shape, off in table:          # every tensor, a few entries each
        k = int(np.prod(shape))
        coords += [off + int(i) for i in rng.choice(k, size=min(k, 4), replace=False)]
    h = 1e-6
    for c in coords:
        tp, tm = theta.copy(), theta.copy()
        tp[c] += h
        tm[c] -= h
        fd = (Mo.loss_only(net, tp, x, y) - Mo.loss_only(net, tm, x, y)) / (2 * h)
        assert abs(fd - g[c]) <= 1e-6 + 1e-5 * abs(g[c]), (arch, c, fd, g[c])
    # padding gaps of the flat layout carry no gradient
    used = np.zeros(total, dtype=bool)
    for name, kind, shape, off in table:
        used[off:off + int(np.prod(shape))] = True
    assert np.all(g[~used] == 0.0)


# ----------------------------------------------------------------------------
# independent float64 implementation with torch autograd
# ----------------------------------------------------------------------------
def _rounder(kind):
    """Rounding to bf16 (via float32, ties to even) or float32, in float64."""
    if kind == "bf16":
        return lambda t: t.to(torch.float32).to(torch.bfloat16).to(torch.float64)
    return lambda t: t.to(torch.float32).to(torch.float64)


def _rounding_functions(kind):
    """Three autograd functions rounding to `kind`: the forward value only,
    the gradient only, or neither (kind None)."""
    if kind is None:
        ident = lambda t: t
        return ident, ident
    rnd = _rounder(kind)

    class ForwardOnly(torch.autograd.Function):
        @staticmethod
        def forward(ctx, x):
            return rnd(x)

        @staticmethod
        def backward(ctx, g):
            return g

    class GradientOnly(torch.autograd.Function):
        @staticmethod
        def forward(ctx, x):
            return x.view_as(x)

        @staticmethod
        def backward(ctx, g):
            return rnd(g)

    return ForwardOnly.apply, GradientOnly.apply


def torch_forward(net, p, x, mode=None):
    """Run `net` with torch ops; p maps names to torch tensors.  mode (the
    oracle's bf16 modes, written independently): "operands" -- every
    convolution and linear contraction reads bf16-rounded operands (inputs and
    weights forward, the output gradient backward; the bias is added after the
    contraction, so its gradient is the unrounded one); "bf16" -- the same,
    and every layer's output (forward) and input gradient (backward) rounded
    to bf16, residual blocks included."""
    op_kind = {"operands": "bf16", "bf16": "bf16"}.get(mode)
    st_kind = mode if mode == "bf16" else None
    R, G = _rounding_functions(op_kind)          # contraction operands
    SF, SG = _rounding_functions(st_kind)        # tensors between layers

    def leaf(mod, h):
        if isinstance(mod, Mo.Conv):
            w = R(p[mod.name + ".weight"]).permute(0, 3, 1, 2)      # OHWI -> OIHW
            out = G(F.conv2d(R(h), w, None, stride=mod.stride, padding=mod.pad))
            if mod.bias:
                out = out + p[mod.name + ".bias"].view(1, -1, 1, 1)
            return out
        if isinstance(mod, Mo.BatchNorm):
            return F.batch_norm(h, None, None, p[mod.name + ".gamma"], p[mod.name + ".beta"],
                                training=True, eps=1e-5)
        if isinstance(mod, Mo.ReLU):
            return F.relu(h)
        if isinstance(mod, Mo.MaxPool2):
            return F.max_pool2d(h, 2)
        if isinstance(mod, Mo.GlobalAvgPool):
            return h.mean(dim=(2, 3))
        if isinstance(mod, Mo.Flatten):
            return h.reshape(h.shape[0], -1)
        if isinstance(mod, Mo.Linear):
            return G(F.linear(R(h), R(p[mod.name + ".weight"]))) + p[mod.name + ".bias"]
        raise TypeError(mod)

    def run(mod, h):
        if isinstance(mod, Mo.Sequential):
            for m in mod.mods:
                h = run(m, h)
            return h
        h = SG(h)          # this layer's input gradient is stored
        if isinstance(mod, Mo.BasicBlock):
            a = run(mod.main, h)
            s = run(mod.short, h) if mod.short else h
            return SF(F.relu(a + s))
        return SF(leaf(mod, h))

    return run(net, x)


def torch_grad(net, table, total, theta, x, y, mode=None, dtype=torch.float64):
    p = {}
    for name, kind, shape, off in table:
        p[name] = torch.tensor(theta[off:off + int(np.prod(shape))].reshape(shape),
                               dtype=dtype, requires_grad=True)
    logits = torch_forward(net, p, torch.tensor(x, dtype=dtype), mode)
    loss = F.cross_entropy(logits, torch.tensor(y, dtype=torch.int64))
    loss.backward()
    loss = loss.detach()
    g = np.zeros(total)
    for name, kind, shape, off in table:
        g[off:off + int(np.prod(shape))] = p[name].grad.double().numpy().ravel()
    return float(loss), g


@pytest.mark.parametrize("arch", sorted(TINY))
def test_against_torch_autograd_small(arch):
    kw, in_shape, n = TINY[arch]
    net, table, total, theta, x, y = rand_problem(arch, kw, in_shape, n, seed=21)
    loss, g = Mo.worker_grad(net, theta, x, y)
    tl, tg = torch_grad(net, table, total, theta, x, y)
    assert abs(loss - tl) < 1e-12 * max(1.0, abs(tl))
    assert np.max(np.abs(g - tg)) <= 1e-11 * np.max(np.abs(tg))


@pytest.mark.parametrize("arch,n", [("mlp", 6), ("small_cnn", 3), ("resnet18", 2), ("resnet50", 1),
                                    ("vgg16", 3)])
def test_against_torch_autograd_full_size(arch, n):
    """The full-size networks of the workloads, He-normal parameters."""
    from paper_2110_08941_amd import synth
    net = Mo.build(arch)
    table, total = Mo.param_table(net)
    theta = synth.he_normal(table, total, seed=3).astype(np.float64)
    x, y = synth.batch((784,) if arch == "mlp" else (3, 32, 32), n, seed=3, step=0)
    loss, g = Mo.worker_grad(net, theta, x, y)
    tl, tg = torch_grad(net, table, total, theta, x, y)
    assert abs(loss - tl) < 1e-11 * max(1.0, abs(tl))
    assert np.max(np.abs(g - tg)) <= 1e-10 * np.max(np.abs(tg))


def test_param_counts():
    """Trainable parameter counts of the four networks (conv weights without
    bias where batch-norm follows)."""
    expect = {"mlp": 784 * 256 + 256 + 256 * 10 + 10,
              "small_cnn": 27 * 32 + 32 + 288 * 64 + 64 + 576 * 128 + 128 + 1280 + 10,
              "resnet18": 11173962, "resnet50": 23520842, "vgg16": 14986698}
    for arch, count in expect.items():
        net = Mo.build(arch)
        assert Mo.true_param_count(net) == count
        # torch's own modules, built independently, agree for the two large ones
    tv = torch.nn
    vgg = tv.Sequential()
    cin = 3
    for v in Mo.VGG16_CFG:
        if v != "M":
            vgg.append(tv.Conv2d(cin, v, 3, padding=1, bias=False))
            vgg.append(tv.BatchNorm2d(v))
            cin = v
    vgg.append(tv.Linear(512, 512))
    vgg.append(tv.Linear(512, 10))
    assert sum(q.numel() for q in vgg.parameters()) == 14986698


@pytest.mark.parametrize("arch", ["mlp", "small_cnn"])
def test_full_batch_invariant(arch):
    """Eq. (1) with weights n_m / N: sum_m (n_m/N) * (mean gradient over
    partition m) is the mean gradient over the whole batch, for any split
    (networks without batch-norm, whose per-sample loss does not depend on
    the other samples)."""
    kw, in_shape, _ = TINY[arch]
    net, table, total, theta, x, y = rand_problem(arch, kw, in_shape, 12, seed=31)
    _, full = Mo.worker_grad(net, theta, x, y)
    for n in ([12], [6, 6], [1, 3, 8], [2, 2, 2, 2, 4], [5, 7]):
        out = S.step(lambda th, xm, ym: Mo.worker_grad(net, th, xm, ym), theta, None, x, y, n,
                     0.1, 0.0, 0.0)
        assert np.max(np.abs(out["gbar"] - full)) <= 1e-13 * max(1.0, np.max(np.abs(full)))


def test_bn_worker_statistics_are_per_partition():
    """With batch-norm the per-worker statistics make the weighted average
    depend on the split (the invariant above does not hold); the M = 1 call is
    the full-batch gradient."""
    kw, in_shape, _ = TINY["resnet18"]
    net, table, total, theta, x, y = rand_problem("resnet18", kw, in_shape, 8, seed=41)
    grad = lambda th, xm, ym: Mo.worker_grad(net, th, xm, ym)
    _, full = grad(theta, x, y)
    one = S.step(grad, theta, None, x, y, [8], 0.1, 0.0, 0.0)["gbar"]
    two = S.step(grad, theta, None, x, y, [4, 4], 0.1, 0.0, 0.0)["gbar"]
    assert np.array_equal(one, full)
    assert np.max(np.abs(two - full)) > 1e-6


def test_driver_model_clock_partitions():
    """Dynamic Partitioning over several windows with the model clock: the
    first window is even (Algorithm 1, t == 0), every later one is in
    proportion to the speeds; the loss goes down on a fixed batch."""
    kw, in_shape, _ = TINY["small_cnn"]
    net, table, total, theta, x, y = rand_problem("small_cnn", kw, in_shape, 16, seed=51)
    grad = lambda th, xm, ym: Mo.worker_grad(net, th, xm, ym)
    speeds = [[1.0, 1.0, 2.0, 4.0]] * 6
    out = S.run(grad, theta, [(x, y)] * 6, speeds, window=2, lr=0.05, mu=0.0, wd=0.0)
    assert out["partitions"][0] == [4, 4, 4, 4] and out["partitions"][1] == [4, 4, 4, 4]
    for t in range(2, 6):
        assert out["partitions"][t] == [2, 2, 4, 8]
    assert out["cps"][0] == [1.0, 1.0, 2.0, 4.0]


def test_maxpool_ties_match_torch():
    """Max-pool backward with tied window entries: the gradient goes to the
    first maximum in row-major window order, as torch's CPU max-pool does."""
    from oracle import layers as L
    rng = np.random.default_rng(8)
    base = rng.integers(0, 3, size=(2, 4, 6, 5)).astype(np.float64)   # many ties
    dy = rng.standard_normal((2, 2, 3, 5))
    xt = torch.tensor(base.transpose(0, 3, 1, 2), requires_grad=True)
    F.max_pool2d(xt, 2).backward(torch.tensor(dy.transpose(0, 3, 1, 2)))
    ref = xt.grad.numpy().transpose(0, 2, 3, 1)
    np.testing.assert_array_equal(L.maxpool2_backward(base, dy), ref)


@pytest.mark.parametrize("mutation", ["bn_drop_term", "conv_flip_tap", "pool_last_max", "ce_no_mean"])
def test_pins_catch_planted_mistakes(monkeypatch, mutation):
    """A plausible mistake planted in the oracle (on the CPU) is caught by the
    autograd comparison above."""
    from oracle import layers as L
    if mutation == "bn_drop_term":
        def bad(dy, gamma, cache):
            xhat, rstd = cache
            axes = tuple(range(dy.ndim - 1))
            count = dy.size // dy.shape[-1]
            db, dg = dy.sum(axis=axes), (dy * xhat).sum(axis=axes)
            return gamma * rstd / count * (count * dy - db), dg, db
        monkeypatch.setattr(L, "bn_backward", bad)
        arch = "resnet18"
    elif mutation == "conv_flip_tap":
        good = L.conv_backward
        def bad(x, w, dy, stride, pad):
            dx, dw, db = good(x, w, dy, stride, pad)
            return dx, dw[:, ::-1, ::-1, :].copy(), db
        monkeypatch.setattr(L, "conv_backward", bad)
        arch = "small_cnn"
    elif mutation == "pool_last_max":
        def bad(x, dy):
            y = L.maxpool2_forward(x)
            dx = np.zeros_like(x)
            for i in (0, 1):
                for j in (0, 1):
                    dx[:, i::2, j::2, :] = np.where(x[:, i::2, j::2, :] == y, dy, 0.0)
            return dx
        monkeypatch.setattr(L, "maxpool2_backward", bad)
        arch = "vgg16"
    else:
        good = L.softmax_ce
        def bad(logits, labels):
            loss, dz = good(logits, labels)
            return loss, dz * logits.shape[0]
        monkeypatch.setattr(L, "softmax_ce", bad)
        arch = "mlp"
    if mutation == "pool_last_max":
        with pytest.raises(AssertionError):
            test_maxpool_ties_match_torch()
        return
    kw, in_shape, n = TINY[arch]
    net, table, total, theta, x, y = rand_problem(arch, kw, in_shape, n, seed=21)
    _, g = Mo.worker_grad(net, theta, x, y)
    _, tg = torch_grad(net, table, total, theta, x, y)
    assert np.max(np.abs(g - tg)) > 1e-6 * np.max(np.abs(tg))


def test_bf16_round_matches_torch():
    """Round-to-nearest-even bf16 of the operand rounding against torch's
    float32 -> bfloat16 conversion (ties, subnormals, large values)."""
    from oracle import layers as L
    rng = np.random.default_rng(12)
    x = np.concatenate([rng.standard_normal(100000) * 10.0 ** rng.integers(-30, 30, 100000),
                        np.array([1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, -1.0 - 2.0 ** -8,
                                  1e-40, -3e-39, 0.0, 3.0e38])]).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(L.bf16_round(x), ref)


@pytest.mark.parametrize("arch", sorted(TINY))
def test_fp32_mode_against_torch_float32(arch):
    """The oracle's fp32 mode is float32 arithmetic: it agrees with torch's
    float32 autograd of the same network, and with the exact gradient, to
    float32 accuracy, and differs from the exact one."""
    kw, in_shape, n = TINY[arch]
    net, table, total, theta, x, y = rand_problem(arch, kw, in_shape, n, seed=23)
    loss, g = Mo.worker_grad(net, theta, x, y, storage="fp32")
    tl, tg = torch_grad(net, table, total, theta, x, y, dtype=torch.float32)
    _, ge = Mo.worker_grad(net, theta, x, y)
    scale = np.max(np.abs(ge))
    assert abs(loss - tl) < 1e-5 * max(1.0, abs(tl))
    assert np.max(np.abs(g - tg)) <= 1e-5 * scale
    assert 0 < np.max(np.abs(g - ge)) <= 1e-5 * scale


def test_rounding_realizations():
    """Another realization of the bf16 rounding (Ctx grid = k > 0) keeps
    bf16's relative error bound (2^-8) on every value and places the errors
    elsewhere: a different result from the same inputs, reproducible per k;
    grid 0 is plain round-to-nearest-even."""
    from oracle import layers as L
    rng = np.random.default_rng(5)
    x = rng.standard_normal(200000) * 10.0 ** rng.integers(-8, 8, 200000)
    np.testing.assert_array_equal(Mo.Ctx("bf16").bf16(x), L.bf16_round(x))
    a = Mo.Ctx("bf16", grid=3).bf16(x)
    b = Mo.Ctx("bf16", grid=3).bf16(x)
    c = Mo.Ctx("bf16", grid=4).bf16(x)
    np.testing.assert_array_equal(a, b)
    assert np.all(np.abs(a - x) <= 2.0 ** -8 * np.abs(x))
    assert np.mean(a != L.bf16_round(x)) > 0.2 and np.mean(a != c) > 0.2
    # error statistics of a realization match plain rounding's
    e0 = np.abs(L.bf16_round(x) - x) / np.abs(x)
    e1 = np.abs(a - x) / np.abs(x)
    assert 0.7 < np.mean(e1) / np.mean(e0) < 1.3
    kw, in_shape, n = TINY["small_cnn"]
    net, table, total, theta, x, y = rand_problem("small_cnn", kw, in_shape, n, seed=23)
    _, ge = Mo.worker_grad(net, theta, x, y)
    _, g0 = Mo.worker_grad(net, theta, x, y, storage="bf16")
    _, g1 = Mo.worker_grad(net, theta, x, y, storage="bf16", grid=1)
    scale = np.max(np.abs(ge))
    assert np.max(np.abs(g0 - g1)) > 0
    assert np.max(np.abs(g1 - ge)) < 20 * max(np.max(np.abs(g0 - ge)), 1e-6 * scale)


@pytest.mark.parametrize("mode", ["operands", "bf16"])
@pytest.mark.parametrize("arch", sorted(TINY))
def test_rounding_modes_against_torch(arch, mode):
    """The oracle's bf16 modes against an independent torch autograd
    implementation that rounds the same values with autograd functions
    (forward value only, gradient only) around each contraction and each
    layer."""
    kw, in_shape, n = TINY[arch]
    net, table, total, theta, x, y = rand_problem(arch, kw, in_shape, n, seed=23)
    loss, g = Mo.worker_grad(net, theta, x, y, storage=mode)
    tl, tg = torch_grad(net, table, total, theta, x, y, mode=mode)
    assert abs(loss - tl) < 1e-12 * max(1.0, abs(tl))
    assert np.max(np.abs(g - tg)) <= 1e-11 * np.max(np.abs(tg))
    # the rounding is really applied: the exact gradient differs
    _, ge = Mo.worker_grad(net, theta, x, y)
    assert np.max(np.abs(g - ge)) > 1e-6 * np.max(np.abs(ge))


def test_decision_toggles():
    """Toggling a listed ambiguous ReLU decision changes the gradient only
    along that decision's direction; toggles are a set; every listed decision
    has a margin below the capture threshold."""
    kw, in_shape, n = TINY["small_cnn"]
    net, table, total, theta, x, y = rand_problem("small_cnn", kw, in_shape, 6, seed=61)
    _, ge = Mo.worker_grad(net, theta, x, y)
    ctx = Mo.Ctx("exact", capture=0.05)
    _, g0 = Mo.worker_grad(net, theta, x, y, ctx=ctx)
    assert np.array_equal(g0, ge)
    assert ctx.ambiguous and all(m < 0.05 for _, _, m in ctx.ambiguous)
    c, i, _ = ctx.ambiguous[0]
    _, g1 = Mo.worker_grad(net, theta, x, y, ctx=Mo.Ctx("exact", toggles={(c, i)}))
    assert np.max(np.abs(g1 - g0)) > 0
    _, g2 = Mo.worker_grad(net, theta, x, y, ctx=Mo.Ctx("exact", toggles={(c, i), (c, i)}))
    assert np.array_equal(g1, g2)


def test_separated_decisions_have_large_margins():
    """The separated batch-norm parameters keep every ReLU input of the BN
    networks well away from zero (the regime of the direct GPU comparisons)."""
    from paper_2110_08941_amd import synth
    for arch in ("resnet18", "resnet50", "vgg16"):
        kw, in_shape, n = TINY[arch]
        net = Mo.build(arch, **kw)
        table, total = Mo.param_table(net)
        theta = synth.separate_decisions(table, synth.he_normal(table, total, 1), 1)
        x, y = synth.batch(in_shape, 6, 1, 0, classes=3)
        ctx = Mo.Ctx("exact")
        Mo.worker_grad(net, theta.astype(np.float64), x, y, ctx=ctx)
        relu = [m[1][0] for m in ctx.margins if m[0] == "relu"]
        assert min(relu) > 1e-3


# ----------------------------------------------------------------------------
# ResNet-50 structure, written independently with torch.nn modules
# ----------------------------------------------------------------------------
class _TorchBottleneck(torch.nn.Module):
    def __init__(self, cin, mid, stride, exp):
        super().__init__()
        tn = torch.nn
        self.conv1, self.bn1 = tn.Conv2d(cin, mid, 1, bias=False), tn.BatchNorm2d(mid)
        self.conv2 = tn.Conv2d(mid, mid, 3, stride=stride, padding=1, bias=False)
        self.bn2 = tn.BatchNorm2d(mid)
        self.conv3, self.bn3 = tn.Conv2d(mid, mid * exp, 1, bias=False), tn.BatchNorm2d(mid * exp)
        self.proj = None
        if stride != 1 or cin != mid * exp:
            self.proj = tn.Conv2d(cin, mid * exp, 1, stride=stride, bias=False)
            self.proj_bn = tn.BatchNorm2d(mid * exp)

    def forward(self, x):
        h = F.relu(self.bn1(self.conv1(x)))
        h = F.relu(self.bn2(self.conv2(h)))
        h = self.bn3(self.conv3(h))
        return F.relu(h + (self.proj_bn(self.proj(x)) if self.proj is not None else x))


class _TorchResNet50(torch.nn.Module):
    """CIFAR ResNet-50 as commonly written for 32x32 inputs: 3x3 stem, stages
    of [3, 4, 6, 3] bottlenecks at inner widths 64..512, expansion 4, stride 2
    on the 3x3 conv of each later stage's first block."""

    def __init__(self, in_ch=3, widths=(64, 128, 256, 512), blocks=(3, 4, 6, 3), exp=4,
                 classes=10):
        super().__init__()
        tn = torch.nn
        self.stem, self.stem_bn = tn.Conv2d(in_ch, widths[0], 3, padding=1, bias=False), \
            tn.BatchNorm2d(widths[0])
        layers, cin = [], widths[0]
        for si, (w, nb) in enumerate(zip(widths, blocks)):
            for bi in range(nb):
                layers.append(_TorchBottleneck(cin, w, 2 if si > 0 and bi == 0 else 1, exp))
                cin = w * exp
        self.layers = tn.ModuleList(layers)
        self.blocks = blocks
        self.fc = tn.Linear(cin, classes)

    def forward(self, x):
        h = F.relu(self.stem_bn(self.stem(x)))
        for b in self.layers:
            h = b(h)
        return self.fc(h.mean(dim=(2, 3)))

    def oracle_names(self):
        """(oracle tensor name, torch parameter) pairs."""
        out = [("stem.weight", self.stem.weight), ("stem_bn.gamma", self.stem_bn.weight),
               ("stem_bn.beta", self.stem_bn.bias)]
        i = 0
        for si, nb in enumerate(self.blocks):
            for bi in range(nb):
                b, pre = self.layers[i], "layer%d.%d." % (si + 1, bi)
                i += 1
                mods = [("conv1", b.conv1), ("bn1", b.bn1), ("conv2", b.conv2), ("bn2", b.bn2),
                        ("conv3", b.conv3), ("bn3", b.bn3)]
                if b.proj is not None:
                    mods += [("proj", b.proj), ("proj_bn", b.proj_bn)]
                for nm, m in mods:
                    if isinstance(m, torch.nn.Conv2d):
                        out.append((pre + nm + ".weight", m.weight))
                    else:
                        out += [(pre + nm + ".gamma", m.weight), (pre + nm + ".beta", m.bias)]
        return out + [("fc.weight", self.fc.weight), ("fc.bias", self.fc.bias)]


def test_resnet50_matches_independent_torch_modules():
    """The oracle's bottleneck network against one built from torch.nn modules
    (training-mode batch-norm): same parameter count at full size; at reduced
    width the same loss and gradient, tensor by tensor, with the oracle's flat
    layout mapped onto the module's parameters by name."""
    full = _TorchResNet50()
    assert sum(q.numel() for q in full.parameters()) == 23520842
    kw, in_shape, n = TINY["resnet50"]
    net, table, total, theta, x, y = rand_problem("resnet50", kw, in_shape, n, seed=71)
    tm = _TorchResNet50(in_ch=3, widths=kw["widths"], blocks=kw["blocks"], exp=kw["expansion"],
                        classes=kw["classes"]).double()
    offs = {name: (off, shape) for name, kind, shape, off in table}
    pairs = tm.oracle_names()
    assert sorted(nm for nm, _ in pairs) == sorted(offs)
    with torch.no_grad():
        for nm, prm in pairs:
            off, shape = offs[nm]
            v = torch.tensor(theta[off:off + int(np.prod(shape))].reshape(shape))
            prm.copy_(v.permute(0, 3, 1, 2) if v.ndim == 4 else v)    # OHWI -> OIHW
    loss_t = F.cross_entropy(tm(torch.tensor(x)), torch.tensor(y, dtype=torch.int64))
    loss_t.backward()
    loss, g = Mo.worker_grad(net, theta, x, y)
    assert abs(loss - float(loss_t.detach())) < 1e-12
    scale = max(float(prm.grad.abs().max()) for _, prm in pairs)
    for nm, prm in pairs:
        off, shape = offs[nm]
        gt = prm.grad.numpy()
        gt = gt.transpose(0, 2, 3, 1) if gt.ndim == 4 else gt
        np.testing.assert_allclose(g[off:off + int(np.prod(shape))].reshape(shape), gt,
                                   rtol=0, atol=1e-11 * scale, err_msg=nm)


def test_bf16_operand_floor():
    """How far bf16 arithmetic alone moves the gradient from the exact one
    (the reason the bf16 GPU tests bound a tensor by 3 x this floor where it
    exceeds 2e-2).  Rounding only the contraction operands to bf16 keeps every
    tensor of the small CNN within 2e-2 of the exact gradient, but moves most
    tensors of the full-width ResNet-18 by more than that, with every ReLU
    decision far from zero (separated batch-norm parameters): through the deep
    batch-norm chain the rounding of the always-on channels' large-mean
    activations is amplified, and batch-norm shift gradients are small residues
    of cancelling sums."""
    from paper_2110_08941_amd import synth
    from tests.gpu_util import pertensor, separate_by_bias
    out = {}
    for arch, n in (("small_cnn", 8), ("resnet18", 4)):
        net = Mo.build(arch)
        table, total = Mo.param_table(net)
        theta = synth.he_normal(table, total, n)
        x, y = synth.batch((3, 32, 32), n, n, 1)
        if arch == "small_cnn":
            theta = separate_by_bias(net, theta, x, table, n)
        else:
            theta = synth.separate_decisions(table, theta, n)
        th = theta.astype(np.float64)
        ctx = Mo.Ctx("exact")
        _, ge = Mo.worker_grad(net, th, x, y, ctx=ctx)
        assert min(m[1][0] for m in ctx.margins if m[0] == "relu" and m[1].size) > 1e-4
        _, go = Mo.worker_grad(net, th, x, y, storage="operands")
        out[arch] = [e for _, e, _ in pertensor(go, ge, table)]
    assert max(out["small_cnn"]) <= 2e-2
    assert sum(e > 2e-2 for e in out["resnet18"]) > len(out["resnet18"]) // 2
