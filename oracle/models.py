"""Networks of the oracle and the per-worker gradient (test infrastructure).

The per-worker gradient is g_m = grad_theta of f_m, the mean loss over
worker m's partition (Section 1, Eq. (1); Section 3 describes each worker
computing the gradient of its mini-batch).  The paper trains ResNet50 and VGG16
on CIFAR10 (Section 5); the networks here are the CIFAR-shaped MLP, small CNN,
ResNet-18 and VGG-16 of the workloads, each buildable at reduced width and
resolution so that finite differences stay cheap.

Flat parameter vector layout (written here independently of the GPU library;
a test checks that both tables agree):
  * tensors in forward order; a layer's bias follows its weight; batch-norm
    stores gamma then beta; in a residual block the order is conv1, bn1,
    conv2, bn2, then the projection conv and its batch-norm;
  * every tensor starts at a multiple of 64 elements; the gaps are zero.
"""
import numpy as np

from . import layers as L

ALIGN = 64


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

    def forward(self, x, p):
        b = p[self.name + ".bias"] if self.bias else None
        return L.conv_forward(x, p[self.name + ".weight"], self.stride, self.pad, b), x

    def backward(self, cache, dy, p, g, need_dx=True):
        x = cache
        dx, dw, db = L.conv_backward(x, p[self.name + ".weight"], dy, self.stride, self.pad)
        g[self.name + ".weight"] += dw
        if self.bias:
            g[self.name + ".bias"] += db
        return dx


class Linear:
    def __init__(self, name, fin, fout):
        self.name, self.fin, self.fout = name, fin, fout

    def params(self):
        return [(self.name + ".weight", "lin_w", (self.fout, self.fin)),
                (self.name + ".bias", "bias", (self.fout,))]

    def forward(self, x, p):
        return L.linear_forward(x, p[self.name + ".weight"], p[self.name + ".bias"]), x

    def backward(self, cache, dy, p, g, need_dx=True):
        dx, dw, db = L.linear_backward(cache, p[self.name + ".weight"], dy)
        g[self.name + ".weight"] += dw
        g[self.name + ".bias"] += db
        return dx


class BatchNorm:
    def __init__(self, name, c):
        self.name, self.c = name, c

    def params(self):
        return [(self.name + ".gamma", "bn_gamma", (self.c,)),
                (self.name + ".beta", "bn_beta", (self.c,))]

    def forward(self, x, p):
        return L.bn_forward(x, p[self.name + ".gamma"], p[self.name + ".beta"])

    def backward(self, cache, dy, p, g, need_dx=True):
        dz, dgamma, dbeta = L.bn_backward(dy, p[self.name + ".gamma"], cache)
        g[self.name + ".gamma"] += dgamma
        g[self.name + ".beta"] += dbeta
        return dz


class ReLU:
    def params(self):
        return []

    def forward(self, x, p):
        y = L.relu_forward(x)
        return y, y

    def backward(self, cache, dy, p, g, need_dx=True):
        return L.relu_backward(cache, dy)


class MaxPool2:
    def params(self):
        return []

    def forward(self, x, p):
        return L.maxpool2_forward(x), x

    def backward(self, cache, dy, p, g, need_dx=True):
        return L.maxpool2_backward(cache, dy)


class GlobalAvgPool:
    def params(self):
        return []

    def forward(self, x, p):
        return L.gap_forward(x), x.shape

    def backward(self, cache, dy, p, g, need_dx=True):
        return L.gap_backward(cache, dy)


class Flatten:
    """NHWC [n,1,1,c] -> [n,c] (only used where h = w = 1, so the order of
    flattening is immaterial)."""

    def params(self):
        return []

    def forward(self, x, p):
        assert x.shape[1] == 1 and x.shape[2] == 1
        return x.reshape(x.shape[0], -1), x.shape

    def backward(self, cache, dy, p, g, need_dx=True):
        return dy.reshape(cache)


class Sequential:
    def __init__(self, mods):
        self.mods = mods

    def params(self):
        out = []
        for m in self.mods:
            out += m.params()
        return out

    def forward(self, x, p):
        caches = []
        for m in self.mods:
            x, c = m.forward(x, p)
            caches.append(c)
        return x, caches

    def backward(self, caches, dy, p, g, need_dx=True):
        for i in range(len(self.mods) - 1, -1, -1):
            dy = self.mods[i].backward(caches[i], dy, p, g, need_dx=(i > 0 or need_dx))
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

    def forward(self, x, p):
        a, ca = self.main.forward(x, p)
        if self.short:
            s, cs = self.short.forward(x, p)
        else:
            s, cs = x, None
        y = L.relu_forward(a + s)
        return y, (ca, cs, y)

    def backward(self, cache, dy, p, g, need_dx=True):
        ca, cs, y = cache
        dpre = L.relu_backward(y, dy)
        dx = self.main.backward(ca, dpre, p, g)
        if self.short:
            dx = dx + self.short.backward(cs, dpre, p, g)
        else:
            dx = dx + dpre
        return dx


# ----------------------------------------------------------------------------
# architectures
# ----------------------------------------------------------------------------
VGG16_CFG = (64, 64, "M", 128, 128, "M", 256, 256, 256, "M", 512, 512, 512, "M",
             512, 512, 512, "M")


def mlp(in_dim=784, hidden=256, classes=10):
    """Linear(in, hidden) + ReLU + Linear(hidden, classes)."""
    return Sequential([Linear("fc1", in_dim, hidden), ReLU(), Linear("fc2", hidden, classes)])


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
    mods += [Flatten(), Linear("fc1", cin, fc_hidden), ReLU(), Linear("fc2", fc_hidden, classes)]
    return Sequential(mods)


ARCHS = {"mlp": mlp, "small_cnn": small_cnn, "resnet18": resnet18, "vgg16": vgg16}


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


def worker_grad(net, theta, x, y):
    """g_m = gradient of f_m = (1/n_m) sum_i CE(net(x_i), y_i) over the worker's
    n_m samples (Eq. (1) with the expectation taken over the partition).
    Batch-norm statistics are those of this worker's samples.
    Returns (loss_m, g_m) with g_m a flat float64 vector in the layout above."""
    table, total = param_table(net)
    th = np.asarray(theta, dtype=np.float64)
    assert th.shape == (total,)
    p = views(th, table)
    g = np.zeros(total, dtype=np.float64)
    gv = views(g, table)
    logits, caches = net.forward(to_nhwc(x), p)
    loss, dz = L.softmax_ce(logits, np.asarray(y, dtype=np.int64))
    net.backward(caches, dz, p, gv, need_dx=False)
    return loss, g


def loss_only(net, theta, x, y):
    table, total = param_table(net)
    p = views(np.asarray(theta, dtype=np.float64), table)
    logits, _ = net.forward(to_nhwc(x), p)
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
