"""Layer definitions of the oracle: forward and backward, NHWC, in the
arithmetic type of their arguments (float64 for the definition; float32 for
the oracle's fp32-arithmetic mode).

Test infrastructure (see the package docstring): plain definitions written
from the textbook formulas, not optimised.  The loss these layers build is the
per-sample loss f(theta; x) of Eq. (1), Section 1 of the paper; the paper fixes
only "image classification with ResNet/VGG networks" (Section 5), so the layer
set is the standard one for those networks.

Layouts:
  activations  x[n, h, w, c]            (channels last)
  conv weight  W[c_out, kh, kw, c_in]   (OHWI)
  linear       W[out, in], b[out]
"""
import numpy as np


# ----------------------------------------------------------------------------
# bf16 rounding (the arithmetic of a bf16 path)
# ----------------------------------------------------------------------------
def bf16_round(x):
    """Nearest bf16 value (8-bit significand), ties to even, of each entry:
    the value is first rounded to float32, then its low 16 bits are rounded
    away; returned as float64."""
    f = np.array(x, dtype=np.float32)
    u = f.view(np.uint32)
    lsb = (u >> 16) & np.uint32(1)
    u += np.uint32(0x7FFF)
    u += lsb
    u &= np.uint32(0xFFFF0000)
    return f.astype(np.float64)


# ----------------------------------------------------------------------------
# convolution
# ----------------------------------------------------------------------------
def conv_out_size(h, k, stride, pad):
    """Output extent of a convolution: floor((h + 2 pad - k) / stride) + 1."""
    return (h + 2 * pad - k) // stride + 1


def conv_forward(x, w, stride, pad, b=None):
    """y[n,o,p,co] = sum_{r,s,ci} xpad[n, o*stride + r, p*stride + s, ci] * W[co,r,s,ci] (+ b[co]).

    Written as one matmul per kernel tap (r, s).
    """
    n, h, wd, ci = x.shape
    co, kh, kw, ci2 = w.shape
    assert ci == ci2
    dt = np.result_type(x, w)
    ho = conv_out_size(h, kh, stride, pad)
    wo = conv_out_size(wd, kw, stride, pad)
    xp = np.zeros((n, h + 2 * pad, wd + 2 * pad, ci), dtype=dt)
    xp[:, pad:pad + h, pad:pad + wd, :] = x
    y = np.zeros((n * ho * wo, co), dtype=dt)
    for r in range(kh):
        for s in range(kw):
            patch = xp[:, r:r + stride * (ho - 1) + 1:stride, s:s + stride * (wo - 1) + 1:stride, :]
            y += np.ascontiguousarray(patch).reshape(-1, ci) @ w[:, r, s, :].T
    y = y.reshape(n, ho, wo, co)
    if b is not None:
        y += b
    return y


def conv_backward(x, w, dy, stride, pad):
    """Gradients of conv_forward: returns (dx, dW, db) for output gradient dy.

    dW[co,r,s,ci] = sum_{n,o,p} dy[n,o,p,co] * xpad[n, o*stride+r, p*stride+s, ci]
    dxpad[n, o*stride+r, p*stride+s, ci] += sum_co dy[n,o,p,co] * W[co,r,s,ci]
    db[co] = sum_{n,o,p} dy[n,o,p,co]
    """
    n, h, wd, ci = x.shape
    co, kh, kw, _ = w.shape
    _, ho, wo, _ = dy.shape
    dt = np.result_type(x, w, dy)
    xp = np.zeros((n, h + 2 * pad, wd + 2 * pad, ci), dtype=dt)
    xp[:, pad:pad + h, pad:pad + wd, :] = x
    dxp = np.zeros_like(xp)
    dw = np.zeros(w.shape, dtype=dt)
    dy2 = np.ascontiguousarray(dy).reshape(-1, co)
    for r in range(kh):
        for s in range(kw):
            rs = (slice(None), slice(r, r + stride * (ho - 1) + 1, stride),
                  slice(s, s + stride * (wo - 1) + 1, stride), slice(None))
            patch = np.ascontiguousarray(xp[rs]).reshape(-1, ci)
            dw[:, r, s, :] = dy2.T @ patch
            dxp[rs] += (dy2 @ w[:, r, s, :]).reshape(n, ho, wo, ci)
    dx = dxp[:, pad:pad + h, pad:pad + wd, :]
    db = dy2.sum(axis=0)
    return dx, dw, db


# ----------------------------------------------------------------------------
# linear
# ----------------------------------------------------------------------------
def linear_forward(x, w, b):
    """y[n,o] = sum_i x[n,i] W[o,i] + b[o]."""
    return x @ w.T + b


def linear_backward(x, w, dy):
    """Returns (dx, dW, db) of linear_forward."""
    return dy @ w, dy.T @ x, dy.sum(axis=0)


# ----------------------------------------------------------------------------
# ReLU
# ----------------------------------------------------------------------------
def relu_forward(x):
    return np.maximum(x, 0.0)


def relu_backward(y, dy):
    """dy * relu'(x) with relu'(0) = 0; the mask is read from the output y = relu(x)."""
    return dy * (y > 0.0)


# ----------------------------------------------------------------------------
# batch normalisation, training mode, statistics over (n, h, w)
# ----------------------------------------------------------------------------
BN_EPS = 1e-5


def bn_forward(z, gamma, beta, eps=BN_EPS):
    """y = gamma * (z - mean) / sqrt(var + eps) + beta, with the batch mean and
    the biased batch variance taken over every axis except the channel axis.
    Returns (y, cache)."""
    axes = tuple(range(z.ndim - 1))
    mean = z.mean(axis=axes)
    var = ((z - mean) ** 2).mean(axis=axes)
    rstd = 1.0 / np.sqrt(var + eps)
    xhat = (z - mean) * rstd
    return gamma * xhat + beta, (xhat, rstd)


def bn_backward(dy, gamma, cache):
    """Backward of bn_forward.  With count = number of reduced elements:
    dbeta = sum dy, dgamma = sum dy*xhat,
    dz = gamma*rstd/count * (count*dy - dbeta - xhat*dgamma)."""
    xhat, rstd = cache
    axes = tuple(range(dy.ndim - 1))
    count = dy.size // dy.shape[-1]
    dbeta = dy.sum(axis=axes)
    dgamma = (dy * xhat).sum(axis=axes)
    dz = gamma * rstd / count * (count * dy - dbeta - xhat * dgamma)
    return dz, dgamma, dbeta


# ----------------------------------------------------------------------------
# pooling
# ----------------------------------------------------------------------------
def maxpool2_forward(x):
    """2x2 max-pool with stride 2 (h and w even)."""
    n, h, w, c = x.shape
    windows = [x[:, i::2, j::2, :] for i in (0, 1) for j in (0, 1)]
    return np.maximum(np.maximum(windows[0], windows[1]), np.maximum(windows[2], windows[3]))


def maxpool2_backward(x, dy):
    """The gradient of each window goes to its first maximum in row-major
    window order (0,0), (0,1), (1,0), (1,1)."""
    y = maxpool2_forward(x)
    dx = np.zeros_like(x)
    taken = np.zeros(y.shape, dtype=bool)
    for i in (0, 1):
        for j in (0, 1):
            hit = (x[:, i::2, j::2, :] == y) & ~taken
            dx[:, i::2, j::2, :] = np.where(hit, dy, 0.0)
            taken |= hit
    return dx


def gap_forward(x):
    """Global average pool: mean over h and w."""
    return x.mean(axis=(1, 2))


def gap_backward(x_shape, dy):
    n, h, w, c = x_shape
    return np.broadcast_to(dy[:, None, None, :] / (h * w), x_shape).copy()


# ----------------------------------------------------------------------------
# softmax cross-entropy, mean over the samples given
# ----------------------------------------------------------------------------
def softmax_ce(logits, labels):
    """L = (1/n) sum_i (logsumexp(z_i) - z_i[y_i]); dz = (softmax(z) - onehot(y)) / n.
    Returns (L, dz)."""
    n = logits.shape[0]
    zmax = logits.max(axis=1, keepdims=True)
    ez = np.exp(logits - zmax)
    sumez = ez.sum(axis=1, keepdims=True)
    lse = np.log(sumez) + zmax
    loss = float(np.mean(lse[:, 0] - logits[np.arange(n), labels]))
    p = ez / sumez
    onehot = np.zeros_like(logits)
    onehot[np.arange(n), labels] = 1.0
    return loss, (p - onehot) / n
