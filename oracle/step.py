"""The synchronous step of the oracle: weighted average, SGD, compute-power
estimate, repartition, and the multi-step driver (test infrastructure).

Readings of the paper taken here (each also listed in the design notes):
  * EDP weighting (Section 4.2): worker m's gradient is weighted by its
    normalised compute power before the exchange.  With the partition sized in
    proportion to compute power (Algorithm 1), the normalised compute power is
    n_m / N up to integer rounding, so the weights used are w_m = n_m / sum n,
    which sum to one; the exchange is then a sum.  With equal partitions this
    is the Sync-SGD mean of Section 1.
  * SGD (Section 1 update, Section 5 momentum 0.9 / weight decay 5e-4):
    d = g + wd*theta; buf = mu*buf + d (buf starts at zero); theta -= lr*buf.
    No dampening, no Nesterov.
  * Repartition (Algorithm 1): the fractional sizes CP_m * N are rounded by
    largest remainder with a pinned order of floating-point operations, ties
    to the lower worker index, and no worker left with zero samples.
"""
import math

import numpy as np


# ----------------------------------------------------------------------------
# exchange and update
# ----------------------------------------------------------------------------
def partition_weights(n):
    """w_m = n_m / sum_j n_j (Section 4.2 with the reading above)."""
    n = np.asarray(n, dtype=np.float64)
    return n / n.sum()


def weighted_average(grads, n):
    """g = sum_m w_m g_m with w_m = n_m / sum n (Section 4.2)."""
    w = partition_weights(n)
    out = np.zeros_like(np.asarray(grads[0], dtype=np.float64))
    for wm, gm in zip(w, grads):
        out += wm * np.asarray(gm, dtype=np.float64)
    return out


def mean_average(grads):
    """g = (1/M) sum_m g_m: the exchange of Sync-SGD and of Dynamic
    Partitioning without the enhancement (Section 5), whatever the partition
    sizes."""
    out = np.zeros_like(np.asarray(grads[0], dtype=np.float64))
    for gm in grads:
        out += np.asarray(gm, dtype=np.float64)
    return out / float(len(grads))


def cosine_lr(lr0, t, total, lr_min=0.0):
    """Cosine annealing (Section 5 names the schedule; SGDR without restarts):
    lr_t = lr_min + (lr0 - lr_min) (1 + cos(pi t / total)) / 2 for step t of
    `total`."""
    return lr_min + (lr0 - lr_min) * (1.0 + math.cos(math.pi * t / total)) / 2.0


def sgd_step(theta, g, buf, lr, mu, wd):
    """One SGD step with momentum and coupled weight decay (Section 1 update
    rule; Section 5 hyper-parameters).  Returns (theta', buf')."""
    theta = np.asarray(theta, dtype=np.float64)
    d = np.asarray(g, dtype=np.float64) + wd * theta
    buf = d.copy() if buf is None else mu * np.asarray(buf, dtype=np.float64) + d
    return theta - lr * buf, buf


# ----------------------------------------------------------------------------
# compute power and repartition
# ----------------------------------------------------------------------------
def estimate_cp(n, xbar):
    """CP_m = |D_m| / X_m (Section 4, Eq. (2)); X_m is the mean time to process
    worker m's mini-batch over the window."""
    return [float(nm) / float(xm) for nm, xm in zip(n, xbar)]


class RepartitionError(ValueError):
    pass


def repartition(cp, total):
    """Algorithm 1, Section 4.1: normalise the compute powers, CP_m /= sum_j CP_j,
    and give worker m a partition of CP_m * |D| samples.

    Pinned arithmetic (IEEE double, no fused operations):
      S   = cp_0 + cp_1 + ... (left to right)
      c_m = cp_m / S                       (normalise)
      q_m = c_m * total                    (fractional size)
      f_m = floor(q_m), r_m = q_m - f_m
      the L = total - sum f_m workers with the largest r_m get one more sample
      (ties: lower index first); then, while some worker has zero samples, one
      sample moves from the largest worker (lowest index on ties) to the
      lowest-index empty worker.
    The even split of the first epoch is repartition([1]*M, total)."""
    m = len(cp)
    if m < 1 or total < m:
        raise RepartitionError("need total >= M >= 1")
    for v in cp:
        if not (isinstance(v, float) or isinstance(v, int)) or not math.isfinite(v) or v <= 0:
            raise RepartitionError("compute powers must be finite and > 0")
    s = 0.0
    for v in cp:
        s = s + float(v)
    q = [(float(v) / s) * float(total) for v in cp]
    f = [math.floor(x) for x in q]
    r = [x - fl for x, fl in zip(q, f)]
    left = total - sum(f)
    if left < 0 or left >= m + 1:
        raise RepartitionError("rounding left %d samples" % left)
    order = sorted(range(m), key=lambda i: (-r[i], i))
    n = list(f)
    for i in order[:left]:
        n[i] += 1
    while 0 in n:
        z = n.index(0)
        big = max(range(m), key=lambda i: (n[i], -i))
        n[big] -= 1
        n[z] += 1
    return n


def even_split(m, total):
    """First epoch of Algorithm 1: CP_m = 1/M for every worker."""
    return repartition([1.0] * m, total)


# ----------------------------------------------------------------------------
# one step and many steps
# ----------------------------------------------------------------------------
def step(net_grad, theta, buf, x, y, n, lr, mu, wd, exchange="edp"):
    """One synchronous step: every worker's gradient on its slice of the batch
    (worker m owns rows [o_m, o_m + n_m), o_m = sum_{j<m} n_j), the exchange
    (exchange="edp": partition-weighted average; "mean": the plain mean), the
    SGD update.  net_grad(theta, x_m, y_m) -> (loss_m, g_m).
    Returns dict with grads, losses, gbar, theta, buf."""
    grads, losses, o = [], [], 0
    for nm in n:
        if nm > 0:
            loss, g = net_grad(theta, x[o:o + nm], y[o:o + nm])
        else:
            loss, g = 0.0, np.zeros(np.shape(theta), dtype=np.float64)
        grads.append(g)
        losses.append(loss)
        o += nm
    gbar = weighted_average(grads, n) if exchange == "edp" else mean_average(grads)
    theta2, buf2 = sgd_step(theta, gbar, buf, lr, mu, wd)
    return {"grads": grads, "losses": losses, "gbar": gbar, "theta": theta2, "buf": buf2}


def smooth_cp(estimator, c, state):
    """Compute power across windows (Section 4.1: the previous epoch only, or a
    history of epochs).  c: this window's estimate n / mean X.  estimator:
    ("window",) -> c; ("ema", alpha) -> alpha c + (1 - alpha) previous (the
    first window: c); ("history", h) -> mean of the last h windows' estimates,
    summed oldest first.  state: dict carried across windows."""
    kind = estimator[0]
    if kind == "window":
        return list(c)
    if kind == "ema":
        alpha = float(estimator[1])
        prev = state.get("prev")
        out = list(c) if prev is None else [alpha * cm + (1.0 - alpha) * pm for cm, pm in zip(c, prev)]
        state["prev"] = out
        return out
    if kind == "history":
        hist = state.setdefault("hist", [])
        hist.append(list(c))
        if len(hist) > int(estimator[1]):
            hist.pop(0)
        out = []
        for j in range(len(c)):
            s = 0.0
            for h in hist:
                s = s + h[j]
            out.append(s / float(len(hist)))
        return out
    raise ValueError("unknown estimator %r" % (estimator,))


def run(net_grad, theta, batches, speeds, window, lr, mu, wd, times=None, n0=None,
        exchange="edp", delays=None, estimator=("window",), lr_total=None, lr_min=0.0,
        theta_store=None):
    """Multi-step driver of Dynamic Partitioning (Algorithm 1).

    batches[t] = (x_t, y_t); speeds[t][m] = s_m at step t.  The time worker m
    needs for its mini-batch at step t is X_m = tau_m / s_m + delay_m, where
    tau_m is the measured device time of its gradient (``times[t][m]``), or,
    without measured times, the model clock X_m = n_m / s_m; delay_m is the
    additive per-batch delay by which Section 5 simulates heterogeneity (none
    by default).  After every ``window`` steps, X_m is averaged over the window
    (summed in step order), c_m = n_m / mean X_m (Eq. (2)), CP =
    smooth_cp(estimator, c) and the next window's partition is repartition(CP,
    N); window = 0 keeps the partition (Sync-SGD).  The first window uses the
    even split (Algorithm 1, t == 0) unless n0 is given.  exchange: "edp"
    (partition-weighted, Section 4.2) or "mean" (Sync-SGD and DP-SGD).  With
    lr_total, step t uses cosine_lr(lr, t, lr_total, lr_min).  Returns dict
    with theta, buf, partitions (per step), losses, cps, xs (X_m per step)."""
    total = int(np.shape(batches[0][1])[0])
    m = len(speeds[0])
    n = list(n0) if n0 is not None else even_split(m, total)
    buf = None
    parts, losses, cps, xs = [], [], [], []
    xsum = [0.0] * m
    state = {}
    for t, (x, y) in enumerate(batches):
        parts.append(list(n))
        lr_t = cosine_lr(lr, t, lr_total, lr_min) if lr_total else lr
        out = step(net_grad, theta, buf, x, y, n, lr_t, mu, wd, exchange)
        theta, buf = out["theta"], out["buf"]
        if theta_store is not None:
            theta, buf = theta_store(theta), theta_store(buf)
        losses.append(out["losses"])
        xt = []
        for j in range(m):
            tau = float(times[t][j]) if times is not None else float(n[j])
            xj = tau / float(speeds[t][j])
            if delays is not None:
                xj = xj + float(delays[j])
            xt.append(xj)
            xsum[j] = xsum[j] + xj
        xs.append(xt)
        if window > 0 and (t + 1) % window == 0:
            xbar = [v / float(window) for v in xsum]
            cp = smooth_cp(estimator, estimate_cp(n, xbar), state)
            cps.append(cp)
            n = repartition(cp, total)
            xsum = [0.0] * m
    return {"theta": theta, "buf": buf, "partitions": parts, "losses": losses,
            "cps": cps, "xs": xs, "next_partition": n}
