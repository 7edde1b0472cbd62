"""Helpers of the GPU parity tests (no arithmetic of the method here)."""
import numpy as np
import pytest
import torch


def require_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2110_08941_amd import hs  # raises if the library is missing
    return hs


def normwise(a, b, den_floor=0.0):
    """max |a - b| / max(max |b|, den_floor) (0 when both are zero)."""
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    den = max(np.max(np.abs(b)) if b.size else 0.0, den_floor)
    num = np.max(np.abs(a - b)) if b.size else 0.0
    if den == 0.0:
        return 0.0 if num == 0.0 else float("inf")
    return float(num / den)


def rne_bf16_bits(x):
    """Round-to-nearest-even bf16 bit pattern of float32 values (finite)."""
    u = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return u.astype(np.uint16)


def bf16_bits_to_f32(b):
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.cuda()


def log(msg):
    print(msg, flush=True)


# ---------------------------------------------------------------------------
# per-tensor error (the normwise measure applied to every parameter tensor)
# ---------------------------------------------------------------------------
TOL = {"fp32": 1e-4, "bf16": 2e-2}
# Where the arithmetic of the path's precision cannot meet the bar on a tensor
# by itself, the bound there is this multiple of the oracle's own error in
# that precision (its "fp32" / "bf16" modes: contraction operands and every
# tensor between layers rounded, sums exact).  A bf16 computation's error is
# one draw from a wide distribution -- over ten realizations of the oracle's
# bf16 rounding (Ctx grid) one VGG-16 tensor's error ranged over 13x -- so the
# bf16 floor is the largest error over REALIZATIONS of that rounding.
FLOOR_FACTOR = 3.0
REALIZATIONS = {"fp32": (0,), "bf16": (0, 1, 2)}
# A tensor whose exact gradient is (numerically) zero -- e.g. every tensor
# below the last batch-norm of a one-sample worker, whose global average pool
# sends the same gradient to every pixel, which the batch-norm then removes --
# has no relative error: a tensor whose largest exact entry is below this
# fraction of the whole vector's largest is measured against that fraction.
ZERO_FLOOR = 1e-3


def pertensor(a, b, table):
    """[(name, max|a - b| / max|b|, max|b|)] for every tensor of the layout
    (rows (name, kind, shape, offset)); the denominator is at least ZERO_FLOOR
    times the largest |b| of the whole vector (numerically zero tensors)."""
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    den_floor = ZERO_FLOOR * (float(np.max(np.abs(b))) if b.size else 0.0)
    out = []
    for row in table:
        name, shape, off = row[0], row[2], row[3]
        k = int(np.prod(shape))
        out.append((name, normwise(a[off:off + k], b[off:off + k], den_floor),
                    float(np.max(np.abs(b[off:off + k]))) if k else 0.0))
    return out


def floor_max(floors):
    """Per-tensor maximum of several pertensor() lists of one layout."""
    out = []
    for rows in zip(*floors):
        out.append(max(rows, key=lambda r: r[1]))
    return out


def oracle_floor(net, theta, x, y, table, exact, dtype):
    """Per-tensor error of the oracle's own arithmetic at the path's precision
    (mode "fp32" or "bf16") against the exact gradient `exact`: the largest
    over the precision's rounding realizations."""
    from oracle import models as Mo
    th = np.asarray(theta, dtype=np.float64)
    out = []
    for k in REALIZATIONS[dtype]:
        out.append(pertensor(Mo.worker_grad(net, th, x, y, storage=dtype, grid=k)[1], exact, table))
        if len(y) > 64:
            log("    floor realization %d of %d done (n=%d)" % (k + 1, len(REALIZATIONS[dtype]), len(y)))
    return floor_max(out)


def check_pertensor(a, b, table, tol, floor=None, what=""):
    """Asserts err_T <= bound_T on every tensor T, with bound_T = tol, or
    max(tol, FLOOR_FACTOR * floor_T) when per-tensor floors (a pertensor()
    list of the same layout) are given.  Logs the worst tensor and how many
    tensors meet tol itself; returns (worst error, its tensor, count within
    tol)."""
    errs = pertensor(a, b, table)
    fl = {name: e for name, e, _ in floor} if floor is not None else {}
    bad, within, worst = [], 0, (0.0, "")
    for name, e, scale in errs:
        bound = max(tol, FLOOR_FACTOR * fl.get(name, 0.0))
        within += e <= tol
        if e > worst[0]:
            worst = (e, name)
        if not e <= bound:
            bad.append("%s %.3e > %.3e (floor %.3e, max|ref| %.2e)"
                       % (name, e, bound, fl.get(name, 0.0), scale))
    msg = "%s: worst tensor %s %.3e; %d of %d tensors within %.0e" % (
        what, worst[1], worst[0], within, len(errs), tol)
    if floor is not None:
        fw = max(floor, key=lambda r: r[1])
        above = sum(1 for _, e, _ in floor if FLOOR_FACTOR * e > tol)
        ratio = max([(e / fl[name], name) for name, e, _ in errs
                     if FLOOR_FACTOR * fl.get(name, 0.0) > tol] or [(0.0, "-")])
        msg += ("; oracle floor worst %s %.3e, %d tensors bounded by 3x floor; "
                "largest error/floor %.2f (%s)" % (fw[0], fw[1], above, ratio[0], ratio[1]))
    log("  " + msg)
    assert not bad, "%s: tensors beyond their bound: %s" % (what, "; ".join(bad[:8]))
    return worst[0], worst[1], within


def separate_by_bias(net, theta, x, table, seed, margin=0.25):
    """BN-free networks (MLP, small CNN): a copy of theta whose ReLU layers'
    biases put every pre-activation of the batch x at least `margin` channel
    standard deviations away from zero (a random half of the channels always
    on, the rest always off), layer by layer in forward order, so that the
    comparison of a bf16 path is free of ambiguous decisions.  Uses the
    oracle's exact forward on x."""
    from oracle import models as Mo
    th = np.array(theta, dtype=np.float64, copy=True)
    rng = np.random.default_rng(seed)
    offs = {row[0]: row[3] for row in table}
    mods = net.mods
    for i, mod in enumerate(mods):
        if not isinstance(mod, Mo.ReLU):
            continue
        prev = mods[i - 1]
        bname = prev.name + ".bias"
        h = Mo.to_nhwc(x)
        p = Mo.views(th, [(r[0], r[1], r[2], r[3]) for r in table])
        ctx = Mo.Ctx("exact")
        for m in mods[:i]:
            h, _ = m.forward(h, p, ctx)
        u = h.reshape(-1, h.shape[-1])
        lo, hi, sd = u.min(axis=0), u.max(axis=0), u.std(axis=0) + 1e-12
        on = rng.random(u.shape[1]) < 0.5
        shift = np.where(on, margin * sd - lo, -(hi + margin * sd))
        th[offs[bname]:offs[bname] + u.shape[1]] += shift
    return th.astype(np.float32)
