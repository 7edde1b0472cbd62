"""Networks of the oracle and the per-worker gradient (test infrastructure).

The per-worker gradient is g_m = grad_theta of f_m, the mean loss over
worker m's partition (Section 1, Eq. (1); Section 3 describes each worker
computing the gradient of its mini-batch).  The paper trains ResNet50 and VGG16
on CIFAR10 (Section 5); the networks here are the CIFAR-shaped MLP, small CNN,
ResNet-18, ResNet-50 and VGG-16 of the workloads, each buildable at reduced
width and resolution so that finite differences stay cheap.

Flat parameter vector layout (written here independently of the GPU library;
a test checks that both tables agree):
  * tensors in forward order; a layer's bias follows its weight; batch-norm
    stores gamma then beta; in a residual block the order is conv1, bn1,
    conv2, bn2 (conv3, bn3 in a bottleneck block), then the projection conv
    and its batch-norm;
  * every tensor starts at a multiple of 64 elements; the gaps are zero.
"""
import numpy as np

from . import layers as L

ALIGN = 64


# ----------------------------------------------------------------------------
# storage precision and decision margins
# ----------------------------------------------------------------------------
class Ctx:
    """Evaluation context of one forward/backward.

    storage = "exact": every value is float64 (the definition).

    The other modes give the error that arithmetic at a lower precision makes
    by itself; a test reads it as the floor of a GPU path's error at that
    precision.  They follow no implementation's storage or fusion choices:
    storage = "operands": every operand of a convolution or linear contraction
    -- the weights, the activations of the forward and weight-gradient
    products, the output gradients of the data- and weight-gradient products
    -- is rounded to bf16 (nearest, ties to even) where the contraction reads
    it; the products are summed in float64; everything else (batch-norm,
    ReLU, pooling, the loss, bias gradients, every stored tensor) stays
    float64.  The bf16 path does this by definition: no bf16 implementation
    has less error.
    storage = "bf16": contraction operands rounded as above, and every tensor
    passed between layers stored in bf16 -- each layer's output in the forward
    pass and each layer's input gradient in the backward pass (residual
    blocks: the block's output and input gradient too).  Sums stay float64
    (bf16 rounding dwarfs the fp32 accumulation of a bf16 path).
    grid = k > 0 (modes "operands" and "bf16"): another realization of the
    same rounding -- every rounded tensor is scaled by 2^u (u uniform in
    [0, 1), drawn per tensor from a generator seeded with k), rounded to bf16
    and scaled back.  Each value keeps the relative error bound of bf16
    rounding (2^-8); where the errors fall changes.  The error of a bf16
    computation is one draw from a wide distribution, so a floor is read as
    the largest error over a few realizations.
    storage = "fp32": the whole pass in float32 arithmetic (numpy float32:
    operands, parameters, every sum and every stored tensor), the arithmetic
    of an fp32 path.

    Every ReLU and max-pool decision records its margin: |pre-activation|
    (ReLU) or the gap between the two largest window values (max-pool),
    relative to the largest magnitude of that tensor.  A decision whose margin
    is within the arithmetic's error is ambiguous: either outcome is correct."""

    MODES = ("exact", "operands", "bf16", "fp32")

    def __init__(self, storage="exact", capture=0.0, toggles=(), grid=0):
        if storage not in self.MODES:
            raise ValueError(storage)
        self.storage = storage
        self.grid = np.random.default_rng(grid) if grid else None
        self.margins = []          # (layer tag, smallest relative margins of the decisions)
        self.capture = capture     # ReLU decisions with a margin below this are listed
        self.ambiguous = []        # (ReLU call index, flat index, margin)
        self.toggles = set(toggles)  # (call index, flat index): backward mask inverted
        self.calls = 0

    def bf16(self, x):
        """x rounded to bf16, on the realization's grid (see grid above)."""
        if self.grid is None:
            return L.bf16_round(x)
        s = 2.0 ** self.grid.random()
        return L.bf16_round(np.asarray(x, dtype=np.float64) * s) / s

    def op(self, x):
        """A contraction operand as the contraction reads it."""
        if self.storage in ("operands", "bf16"):
            return self.bf16(x)
        if self.storage == "fp32":
            return np.asarray(x, dtype=np.float32)
        return x

    def store(self, x):
        """A tensor passed from one layer to the next."""
        if self.storage == "bf16":
            return self.bf16(x)
        if self.storage == "fp32":
            return np.asarray(x, dtype=np.float32)
        return x

    def param(self, x):
        """A parameter read outside a contraction (bias, batch-norm scale and
        shift): float32 in the fp32 mode, else as given."""
        return np.asarray(x, dtype=np.float32) if self.storage == "fp32" else x

    def record(self, tag, rel):
        self.margins.append((tag, np.sort(np.asarray(rel, dtype=np.float64).ravel())[:64]))

    def relu_decide(self, x):
        """Forward ReLU decision on x: records margins, returns (y, call index)."""
        call = self.calls
        self.calls += 1
        rel = relu_margins(x)
        self.record("relu", rel)
        if self.capture > 0.0:
            flat = rel.ravel()
            for i in np.flatnonzero(flat < self.capture):
                self.ambiguous.append((call, int(i), float(flat[i])))
        return L.relu_forward(x), call

    def relu_mask_grad(self, call, y, dy):
        """Backward of the ReLU of call `call`: dy * [y > 0], with the masks of
        the toggled decisions inverted (the other outcome of an ambiguous
        decision; the forward value there is within the margin of zero)."""
        mask = (y > 0.0)
        tog = [i for (c, i) in self.toggles if c == call]
        if tog:
            mask = mask.copy()
            flat = mask.reshape(-1)
            flat[tog] = ~flat[tog]
        return dy * mask

    def min_margin(self):
        vals = [m[1][0] for m in self.margins if m[1].size]
        return min(vals) if vals else float("inf")

    def count_below(self, delta):
        return int(sum(np.count_nonzero(m[1] < delta) for m in self.margins))


def relu_margins(x):
    """|x| / max|x| over the entries (a ReLU decision is x > 0)."""
    scale = np.max(np.abs(x))
    return np.abs(x) / scale if scale > 0 else np.full(x.shape, np.inf)


def pool_margins(x):
    """(largest - second largest) / max|x| of every 2x2 window whose maximum
    is positive (windows of zeros feed a zero ReLU gradient either way)."""
    w = np.stack([x[:, i::2, j::2, :] for i in (0, 1) for j in (0, 1)], axis=-1)
    w = np.sort(w, axis=-1)
    gap = w[..., 3] - w[..., 2]
    scale = np.max(np.abs(x))
    live = w[..., 3] > 0
    return (gap[live] / scale) if scale > 0 else np.array([np.inf])


# ----------------------------------------------------------------------------
# modules
# ----------------------------------------------------------------------------
class Conv:
    def __init__(self, name, cin, cout, k, stride, pad, bias):
        self.name, self.cin, self.cout, self.k = name, cin, cout, k
        self.stride, self.pad, self.bias = stride, pad, bias

    def params(self):
        out = [(self.name + ".weight", "conv_w", (self.cout, self.k, self.k, self.cin))]
        if self.bias:
            out.append((self.name + ".bias", "bias", (self.cout,)))
        return out

    def forward(self, x, p, ctx):
        b = ctx.param(p[self.name + ".bias"]) if self.bias else None
        w = ctx.op(p[self.name + ".weight"])
        return L.conv_forward(ctx.op(x), w, self.stride, self.pad, b), x

    def backward(self, cache, dy, p, g, ctx):
        x = cache
        w = ctx.op(p[self.name + ".weight"])
        dx, dw, _ = L.conv_backward(ctx.op(x), w, ctx.op(dy), self.stride, self.pad)
        g[self.name + ".weight"] += dw
        if self.bias:
            g[self.name + ".bias"] += dy.sum(axis=(0, 1, 2))
        return dx


class Linear:
    def __init__(self, name, fin, fout):
        self.name, self.fin, self.fout = name, fin, fout

    def params(self):
        return [(self.name + ".weight", "lin_w", (self.fout, self.fin)),
                (self.name + ".bias", "bias", (self.fout,))]

    def forward(self, x, p, ctx):
        y = L.linear_forward(ctx.op(x), ctx.op(p[self.name + ".weight"]),
                             ctx.param(p[self.name + ".bias"]))
        return y, x

    def backward(self, cache, dy, p, g, ctx):
        dx, dw, _ = L.linear_backward(ctx.op(cache), ctx.op(p[self.name + ".weight"]), ctx.op(dy))
        g[self.name + ".weight"] += dw
        g[self.name + ".bias"] += dy.sum(axis=0)
        return dx


class BatchNorm:
    def __init__(self, name, c):
        self.name, self.c = name, c

    def params(self):
        return [(self.name + ".gamma", "bn_gamma", (self.c,)),
                (self.name + ".beta", "bn_beta", (self.c,))]

    def forward(self, x, p, ctx):
        y, cache = L.bn_forward(x, ctx.param(p[self.name + ".gamma"]),
                                ctx.param(p[self.name + ".beta"]))
        return y, cache

    def backward(self, cache, dy, p, g, ctx):
        dz, dgamma, dbeta = L.bn_backward(dy, ctx.param(p[self.name + ".gamma"]), cache)
        g[self.name + ".gamma"] += dgamma
        g[self.name + ".beta"] += dbeta
        return dz


class ReLU:
    def params(self):
        return []

    def forward(self, x, p, ctx):
        y, call = ctx.relu_decide(x)
        return y, (y, call)

    def backward(self, cache, dy, p, g, ctx):
        y, call = cache
        return ctx.relu_mask_grad(call, y, dy)


class MaxPool2:
    def params(self):
        return []

    def forward(self, x, p, ctx):
        ctx.record("maxpool", pool_margins(x))
        return L.maxpool2_forward(x), x

    def backward(self, cache, dy, p, g, ctx):
        return L.maxpool2_backward(cache, dy)


class GlobalAvgPool:
    def params(self):
        return []

    def forward(self, x, p, ctx):
        return L.gap_forward(x), x.shape

    def backward(self, cache, dy, p, g, ctx):
        return L.gap_backward(cache, dy)


class Flatten:
    """NHWC [n,1,1,c] -> [n,c] (only used where h = w = 1, so the order of
    flattening is immaterial)."""

    def params(self):
        return []

    def forward(self, x, p, ctx):
        assert x.shape[1] == 1 and x.shape[2] == 1
        return x.reshape(x.shape[0], -1), x.shape

    def backward(self, cache, dy, p, g, ctx):
        return dy.reshape(cache)


class Sequential:
    def __init__(self, mods):
        self.mods = mods

    def params(self):
        out = []
        for m in self.mods:
            out += m.params()
        return out

    def forward(self, x, p, ctx):
        caches = []
        for m in self.mods:
            x, c = m.forward(x, p, ctx)
            x = ctx.store(x)
            caches.append(c)
        return x, caches

    def backward(self, caches, dy, p, g, ctx):
        for i in range(len(self.mods) - 1, -1, -1):
            dy = ctx.store(self.mods[i].backward(caches[i], dy, p, g, ctx))
        return dy


class BasicBlock:
    """out = relu(bn2(conv2(relu(bn1(conv1(x))))) + shortcut(x)); the
    shortcut is the identity, or a 1x1 strided conv + batch-norm when the
    stride or the width changes."""

    def __init__(self, name, cin, cout, stride):
        self.main = Sequential([Conv(name + ".conv1", cin, cout, 3, stride, 1, False),
                                BatchNorm(name + ".bn1", cout), ReLU(),
                                Conv(name + ".conv2", cout, cout, 3, 1, 1, False),
                                BatchNorm(name + ".bn2", cout)])
        self.short = None
        if stride != 1 or cin != cout:
            self.short = Sequential([Conv(name + ".proj", cin, cout, 1, stride, 0, False),
                                     BatchNorm(name + ".proj_bn", cout)])

    def params(self):
        return self.main.params() + (self.short.params() if self.short else [])

    def forward(self, x, p, ctx):
        a, ca = self.main.forward(x, p, ctx)
        if self.short:
            s, cs = self.short.forward(x, p, ctx)
        else:
            s, cs = x, None
        y, call = ctx.relu_decide(a + s)
        y = ctx.store(y)
        return y, (ca, cs, y, call)

    def backward(self, cache, dy, p, g, ctx):
        ca, cs, y, call = cache
        dpre = ctx.relu_mask_grad(call, y, dy)
        dx = self.main.backward(ca, dpre, p, g, ctx)
        if self.short:
            dx = dx + self.short.backward(cs, dpre, p, g, ctx)
        else:
            dx = dx + dpre
        return ctx.store(dx)


class Bottleneck(BasicBlock):
    """out = relu(bn3(conv3(relu(bn2(conv2(relu(bn1(conv1(x)))))))) + shortcut(x)):
    1x1 conv to the block's inner width, 3x3 conv at that width (carrying the
    block's stride), 1x1 conv to expansion x the inner width; the shortcut is
    the identity, or a 1x1 strided conv + batch-norm when the stride or the
    width changes.  Parameter order: conv1, bn1, conv2, bn2, conv3, bn3, then
    the projection conv and its batch-norm."""

    def __init__(self, name, cin, mid, stride, expansion=4):
        cout = mid * expansion
        self.main = Sequential([Conv(name + ".conv1", cin, mid, 1, 1, 0, False),
                                BatchNorm(name + ".bn1", mid), ReLU(),
                                Conv(name + ".conv2", mid, mid, 3, stride, 1, False),
                                BatchNorm(name + ".bn2", mid), ReLU(),
                                Conv(name + ".conv3", mid, cout, 1, 1, 0, False),
                                BatchNorm(name + ".bn3", cout)])
        self.short = None
        if stride != 1 or cin != cout:
            self.short = Sequential([Conv(name + ".proj", cin, cout, 1, stride, 0, False),
                                     BatchNorm(name + ".proj_bn", cout)])


# ----------------------------------------------------------------------------
# architectures
# ----------------------------------------------------------------------------
VGG16_CFG = (64, 64, "M", 128, 128, "M", 256, 256, 256, "M", 512, 512, 512, "M",
             512, 512, 512, "M")


def mlp(in_dim=784, hidden=256, classes=10):
    """Linear(in, hidden) + ReLU + Linear(hidden, classes)."""
    return Sequential([Linear("fc1", in_dim, hidden), ReLU(),
                       Linear("fc2", hidden, classes)])


def small_cnn(in_ch=3, widths=(32, 64, 128), classes=10):
    """conv3x3(+bias) ReLU, conv3x3 ReLU, maxpool2, conv3x3 ReLU, global
    average pool, linear."""
    c1, c2, c3 = widths
    return Sequential([Conv("conv1", in_ch, c1, 3, 1, 1, True), ReLU(),
                       Conv("conv2", c1, c2, 3, 1, 1, True), ReLU(), MaxPool2(),
                       Conv("conv3", c2, c3, 3, 1, 1, True), ReLU(),
                       GlobalAvgPool(), Linear("fc", c3, classes)])


def resnet18(in_ch=3, widths=(64, 128, 256, 512), blocks=(2, 2, 2, 2), classes=10):
    """CIFAR ResNet-18: 3x3 stem conv + BN + ReLU (no max-pool), stages of
    basic blocks (stride 2 at the first block of every stage after the first),
    global average pool, linear."""
    mods = [Conv("stem", in_ch, widths[0], 3, 1, 1, False), BatchNorm("stem_bn", widths[0]), ReLU()]
    cin = widths[0]
    for si, (w, nb) in enumerate(zip(widths, blocks)):
        for bi in range(nb):
            stride = 2 if (si > 0 and bi == 0) else 1
            mods.append(BasicBlock("layer%d.%d" % (si + 1, bi), cin, w, stride))
            cin = w
    mods += [GlobalAvgPool(), Linear("fc", cin, classes)]
    return Sequential(mods)


def resnet50(in_ch=3, widths=(64, 128, 256, 512), blocks=(3, 4, 6, 3), expansion=4, classes=10):
    """CIFAR ResNet-50 (the paper's compute-heavy model, Section 5): 3x3 stem
    conv + BN + ReLU (no max-pool), stages of bottleneck blocks of inner width
    widths[i] and output width expansion x widths[i] (stride 2 on the 3x3 conv
    of the first block of every stage after the first), global average pool,
    linear."""
    mods = [Conv("stem", in_ch, widths[0], 3, 1, 1, False), BatchNorm("stem_bn", widths[0]), ReLU()]
    cin = widths[0]
    for si, (w, nb) in enumerate(zip(widths, blocks)):
        for bi in range(nb):
            stride = 2 if (si > 0 and bi == 0) else 1
            mods.append(Bottleneck("layer%d.%d" % (si + 1, bi), cin, w, stride, expansion))
            cin = w * expansion
    mods += [GlobalAvgPool(), Linear("fc", cin, classes)]
    return Sequential(mods)


def vgg16(in_ch=3, cfg=VGG16_CFG, fc_hidden=512, classes=10):
    """VGG-16 for 32x32 inputs: conv3x3 (no bias) + BN + ReLU per width entry,
    2x2 max-pool per 'M'; then Linear(c, hidden) + ReLU + Linear(hidden,
    classes).  The last pool leaves a 1x1 map."""
    mods, cin, i = [], in_ch, 0
    for v in cfg:
        if v == "M":
            mods.append(MaxPool2())
        else:
            i += 1
            mods += [Conv("conv%d" % i, cin, v, 3, 1, 1, False), BatchNorm("bn%d" % i, v), ReLU()]
            cin = v
    mods += [Flatten(), Linear("fc1", cin, fc_hidden), ReLU(),
             Linear("fc2", fc_hidden, classes)]
    return Sequential(mods)


ARCHS = {"mlp": mlp, "small_cnn": small_cnn, "resnet18": resnet18, "resnet50": resnet50,
         "vgg16": vgg16}


def build(arch, **kw):
    return ARCHS[arch](**kw)


# ----------------------------------------------------------------------------
# flat parameter layout
# ----------------------------------------------------------------------------
def param_table(net):
    """List of (name, kind, shape, offset) and the padded total P."""
    table, off = [], 0
    for name, kind, shape in net.params():
        off = (off + ALIGN - 1) // ALIGN * ALIGN
        table.append((name, kind, tuple(shape), off))
        off += int(np.prod(shape))
    total = (off + ALIGN - 1) // ALIGN * ALIGN
    return table, total


def true_param_count(net):
    return sum(int(np.prod(s)) for _, _, s in net.params())


def views(flat, table):
    """Dict name -> view of the flat vector with the tensor's shape."""
    return {name: flat[off:off + int(np.prod(shape))].reshape(shape)
            for name, _, shape, off in table}


# ----------------------------------------------------------------------------
# per-worker loss and gradient
# ----------------------------------------------------------------------------
def to_nhwc(x):
    """Inputs arrive as NCHW images [n,c,h,w] or flat vectors [n,d]."""
    x = np.asarray(x, dtype=np.float64)
    return x.transpose(0, 2, 3, 1) if x.ndim == 4 else x


def worker_grad(net, theta, x, y, storage="exact", ctx=None, grid=0):
    """g_m = gradient of f_m = (1/n_m) sum_i CE(net(x_i), y_i) over the worker's
    n_m samples (Eq. (1) with the expectation taken over the partition).
    Batch-norm statistics are those of this worker's samples.
    storage: "exact" (float64 throughout), or "operands", "bf16", "fp32"
    (see Ctx; grid selects a rounding realization).  Pass a Ctx to
    read the decision margins afterwards.
    Returns (loss_m, g_m) with g_m a flat float64 vector in the layout above."""
    ctx = ctx or Ctx(storage, grid=grid)
    table, total = param_table(net)
    th = np.asarray(theta, dtype=np.float64)
    assert th.shape == (total,)
    p = views(th, table)
    g = np.zeros(total, dtype=np.float64)
    gv = views(g, table)
    logits, caches = net.forward(to_nhwc(x), p, ctx)
    loss, dz = L.softmax_ce(logits, np.asarray(y, dtype=np.int64))
    net.backward(caches, dz, p, gv, ctx)
    return loss, g


def loss_only(net, theta, x, y, storage="exact"):
    ctx = Ctx(storage)
    table, total = param_table(net)
    p = views(np.asarray(theta, dtype=np.float64), table)
    logits, _ = net.forward(to_nhwc(x), p, ctx)
    loss, _ = L.softmax_ce(logits, np.asarray(y, dtype=np.int64))
    return loss


def forward_flops(net, in_shape):
    """Multiply-accumulates of one forward pass of one sample (dense taps),
    counted by walking the layers; used for the oracle's throughput report."""
    macs = 0
    x = np.zeros((1,) + tuple(in_shape))

    def walk(mod, shape):
        nonlocal macs
        if isinstance(mod, Sequential):
            for m in mod.mods:
                shape = walk(m, shape)
            return shape
        if isinstance(mod, BasicBlock):
            out = walk(mod.main, shape)
            if mod.short:
                walk(mod.short, shape)
            return out
        if isinstance(mod, Conv):
            n, h, w, c = shape
            ho = L.conv_out_size(h, mod.k, mod.stride, mod.pad)
            wo = L.conv_out_size(w, mod.k, mod.stride, mod.pad)
            macs += ho * wo * mod.cout * mod.k * mod.k * mod.cin
            return (n, ho, wo, mod.cout)
        if isinstance(mod, Linear):
            macs += mod.fin * mod.fout
            return (shape[0], mod.fout)
        if isinstance(mod, MaxPool2):
            n, h, w, c = shape
            return (n, h // 2, w // 2, c)
        if isinstance(mod, GlobalAvgPool):
            return (shape[0], shape[3])
        if isinstance(mod, Flatten):
            return (shape[0], int(np.prod(shape[1:])))
        return shape

    walk(net, x.shape if len(in_shape) == 1 else (1, in_shape[1], in_shape[2], in_shape[0]))
    return macs
