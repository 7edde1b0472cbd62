"""Pins of the oracle's exchange, update and repartition (CPU only).

Each test checks the oracle against something other than its own code: hand
-worked examples, closed forms, exact rational arithmetic, or invariants that
Algorithm 1 and Eqs. (2)-(3) fix.
"""
import math
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import step as S

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "repartition_cases.txt")


def load_cases():
    cases = []
    with open(GOLDEN) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            a, b, c = [p.strip() for p in line.split("|")]
            cases.append(([float(v) for v in a.split()], int(b), [int(v) for v in c.split()]))
    return cases


@pytest.mark.parametrize("cp,total,expected", load_cases())
def test_repartition_worked_examples(cp, total, expected):
    assert S.repartition(cp, total) == expected


def exact_largest_remainder(cp, total):
    """Largest remainder in exact rational arithmetic (ties to lower index),
    then the at-least-one-sample rule."""
    fr = [Fraction(v) for v in cp]
    s = sum(fr)
    q = [v / s * total for v in fr]
    f = [math.floor(x) for x in q]
    r = [x - fl for x, fl in zip(q, f)]
    order = sorted(range(len(cp)), key=lambda i: (-r[i], i))
    n = list(f)
    for i in order[:total - sum(f)]:
        n[i] += 1
    while 0 in n:
        z = n.index(0)
        big = max(range(len(n)), key=lambda i: (n[i], -i))
        n[big] -= 1
        n[z] += 1
    return n


def test_repartition_matches_exact_arithmetic():
    """Random integer compute powers whose sum is a power of two, with N a
    power of two: every float operation of the pinned pipeline is then exact,
    so it must equal exact rational arithmetic, ties included.  Other inputs
    (sums not a power of two) must agree wherever the exact remainders are not
    within 1e-9 of a tie."""
    rng = np.random.default_rng(5)
    for _ in range(400):
        m = int(rng.integers(1, 17))
        total = int(2 ** rng.integers(max(1, math.ceil(math.log2(m))), 13))
        cp = [float(rng.integers(1, 64)) for _ in range(m - 1)]
        target = 2.0 ** math.ceil(math.log2(sum(cp) + 1))
        cp.append(target - sum(cp))
        assert S.repartition(cp, total) == exact_largest_remainder(cp, total)
    checked = 0
    for _ in range(400):
        m = int(rng.integers(2, 17))
        total = int(rng.integers(m, 5000))
        cp = [float(v) for v in rng.uniform(0.1, 10.0, size=m)]
        fr = [Fraction(v) for v in cp]
        r = sorted(float((v / sum(fr) * total) % 1) for v in fr)
        if min(b - a for a, b in zip(r, r[1:])) < 1e-9:
            continue
        checked += 1
        assert S.repartition(cp, total) == exact_largest_remainder(cp, total)
    assert checked > 300


def test_repartition_properties():
    """Sum is N; each size within one of its exact share (no fix-up needed
    here); scale invariance by powers of two; a partition is a fixed point."""
    rng = np.random.default_rng(7)
    for _ in range(400):
        m = int(rng.integers(1, 17))
        total = int(rng.integers(m * 8, 5000))
        cp = list(np.exp(rng.normal(0.0, 0.7, size=m)))
        n = S.repartition(cp, total)
        assert sum(n) == total
        s = sum(cp)
        for nm, c in zip(n, cp):
            assert abs(nm - total * c / s) < 1.0 + 1e-9
        k = int(rng.integers(-8, 9))
        assert S.repartition([c * 2.0 ** k for c in cp], total) == n
        assert S.repartition([float(v) for v in n], total) == n


def test_eq3_predicted_times_equalised():
    """Eq. (3): with partitions in proportion to CP, the predicted times
    X'_m = n'_m / CP_m all lie within 1/CP_m of the common value N / sum CP."""
    rng = np.random.default_rng(9)
    for _ in range(200):
        m = int(rng.integers(2, 9))
        total = int(rng.integers(64, 4096))
        cp = list(rng.uniform(0.5, 8.0, size=m))
        n = S.repartition(cp, total)
        common = total / sum(cp)
        for nm, c in zip(n, cp):
            assert abs(nm / c - common) < 1.0 / c + 1e-9


def test_eq2_cp_and_model_clock():
    """Eq. (2): CP_m = |D_m| / X_m.  With the model clock X_m = n_m / s_m the
    estimate returns the speeds, so the repartition is proportional to them."""
    n = [128, 128, 128, 128]
    s = [1.0, 1.0, 2.0, 4.0]
    cp = S.estimate_cp(n, [nm / sm for nm, sm in zip(n, s)])
    assert cp == s
    assert S.repartition(cp, 512) == [64, 64, 128, 256]


def test_repartition_rejects_bad_input():
    for cp, total in [([1.0, float("nan")], 8), ([1.0, 0.0], 8), ([1.0, -1.0], 8),
                      ([1.0, float("inf")], 8), ([1.0, 1.0, 1.0], 2), ([], 4)]:
        with pytest.raises(S.RepartitionError):
            S.repartition(cp, total)


def test_even_split_first_epoch():
    """Algorithm 1 at t == 0: CP_m = 1/M, the first N mod M workers one larger."""
    for m in range(1, 17):
        for total in (m, 2 * m + 3, 1000):
            n = S.even_split(m, total)
            assert n == [total // m + (1 if i < total % m else 0) for i in range(m)]


def test_weighted_average_special_cases():
    """Equal partitions give the Sync-SGD mean (1/M) sum g_m of Section 1; a
    worker with an empty partition contributes nothing; weights sum to one."""
    rng = np.random.default_rng(3)
    g = [rng.standard_normal(50) for _ in range(4)]
    np.testing.assert_allclose(S.weighted_average(g, [8, 8, 8, 8]), sum(g) / 4, rtol=0, atol=1e-15)
    np.testing.assert_allclose(S.weighted_average(g, [0, 3, 0, 1]), 0.75 * g[1] + 0.25 * g[3],
                               rtol=0, atol=1e-15)
    assert abs(S.partition_weights([3, 5, 7]).sum() - 1.0) < 1e-15


def test_sgd_closed_form():
    """From zero momentum, theta' = theta - lr (g + wd theta); a second step
    uses buf2 = mu d1 + d2."""
    rng = np.random.default_rng(4)
    th, g1, g2 = (rng.standard_normal(64) for _ in range(3))
    lr, mu, wd = 0.1, 0.9, 5e-4
    t1, b1 = S.sgd_step(th, g1, None, lr, mu, wd)
    d1 = g1 + wd * th
    np.testing.assert_allclose(t1, th - lr * d1, rtol=0, atol=1e-15)
    t2, b2 = S.sgd_step(t1, g2, b1, lr, mu, wd)
    d2 = g2 + wd * t1
    np.testing.assert_allclose(b2, mu * d1 + d2, rtol=0, atol=1e-15)
    np.testing.assert_allclose(t2, t1 - lr * (mu * d1 + d2), rtol=0, atol=1e-15)
    # plain SGD (mu = 0, wd = 0) is the Section 1 update theta - lr g
    t0, _ = S.sgd_step(th, g1, None, lr, 0.0, 0.0)
    np.testing.assert_allclose(t0, th - lr * g1, rtol=0, atol=1e-15)


def test_sgd_against_torch_optim():
    """Three momentum steps of the oracle's SGD against torch.optim.SGD with the
    Section 5 hyper-parameters (momentum 0.9, weight decay 5e-4, lr 0.1; no
    dampening, no Nesterov), float64, on changing gradients; also plain SGD."""
    import torch
    rng = np.random.default_rng(14)
    for mu, wd in ((0.9, 5e-4), (0.0, 0.0), (0.9, 0.0), (0.0, 5e-4)):
        th0 = rng.standard_normal(257)
        grads = [rng.standard_normal(257) for _ in range(3)]
        p = torch.nn.Parameter(torch.tensor(th0, dtype=torch.float64))
        opt = torch.optim.SGD([p], lr=0.1, momentum=mu, weight_decay=wd, dampening=0.0,
                              nesterov=False)
        th, buf = th0.copy(), None
        for g in grads:
            p.grad = torch.tensor(g, dtype=torch.float64)
            opt.step()
            th, buf = S.sgd_step(th, g, buf, 0.1, mu, wd)
            np.testing.assert_allclose(th, p.detach().numpy(), rtol=0, atol=1e-14)
            if mu != 0.0:
                np.testing.assert_allclose(buf, opt.state[p]["momentum_buffer"].numpy(),
                                           rtol=0, atol=1e-14)


# ----------------------------------------------------------------------------
# Sync-SGD / DP-SGD exchange, estimators across windows, cosine schedule,
# additive delays (Section 5 comparison)
# ----------------------------------------------------------------------------
def _quad_grad(theta, x, y):
    """Per-worker loss (1/n) sum_i 0.5 ||theta - x_i||^2; gradient theta - mean x_i."""
    d = theta[None, :] - x
    return 0.5 * float((d * d).sum()) / len(x), d.mean(axis=0)


def test_edp_weighting_recovers_full_batch_gradient():
    """With per-worker mean gradients, weights n_m / N give exactly the gradient
    of the whole batch (the reason for the Section 4.2 weighting); the plain mean
    does so only for equal partitions."""
    rng = np.random.default_rng(11)
    theta = rng.standard_normal(5)
    x = rng.standard_normal((12, 5))
    y0 = np.zeros(12, dtype=np.int64)
    n = [7, 3, 2]
    full = theta - x.mean(axis=0)
    edp = S.step(_quad_grad, theta, None, x, y0, n, 0.1, 0.0, 0.0, "edp")
    mean = S.step(_quad_grad, theta, None, x, y0, n, 0.1, 0.0, 0.0, "mean")
    np.testing.assert_allclose(edp["gbar"], full, rtol=0, atol=1e-14)
    per = [theta - x[0:7].mean(0), theta - x[7:10].mean(0), theta - x[10:12].mean(0)]
    np.testing.assert_allclose(mean["gbar"], (per[0] + per[1] + per[2]) / 3, rtol=0, atol=1e-14)
    assert np.abs(mean["gbar"] - full).max() > 1e-3
    eq = [4, 4, 4]
    a = S.step(_quad_grad, theta, None, x, y0, eq, 0.1, 0.0, 0.0, "edp")["gbar"]
    b = S.step(_quad_grad, theta, None, x, y0, eq, 0.1, 0.0, 0.0, "mean")["gbar"]
    np.testing.assert_allclose(a, full, rtol=0, atol=1e-14)
    np.testing.assert_allclose(b, full, rtol=0, atol=1e-14)


def test_mean_average_closed_form():
    g = [np.full(3, 1.0), np.full(3, 2.0), np.full(3, 6.0)]
    np.testing.assert_array_equal(S.mean_average(g), np.full(3, 3.0))


def test_cosine_lr_closed_forms():
    """Cosine annealing: lr0 at t = 0, lr_min at t = T, the midpoint at T / 2,
    symmetric about T / 2 and non-increasing."""
    lr0, lmin, T = 0.1, 0.001, 40
    assert S.cosine_lr(lr0, 0, T, lmin) == lr0
    assert abs(S.cosine_lr(lr0, T, T, lmin) - lmin) < 1e-17
    assert abs(S.cosine_lr(lr0, T // 2, T, lmin) - (lr0 + lmin) / 2) < 1e-16
    v = [S.cosine_lr(lr0, t, T, lmin) for t in range(T + 1)]
    assert all(a >= b for a, b in zip(v, v[1:]))
    for t in range(T + 1):
        assert abs(v[t] + v[T - t] - (lr0 + lmin)) < 1e-16
    assert abs(S.cosine_lr(1.0, 1, 3) - 0.75) < 1e-16        # (1 + cos(pi/3)) / 2


def test_smooth_cp_special_cases_and_worked_examples():
    """EMA with alpha = 1 and a history of 1 are the single-window estimate;
    a constant estimate is a fixed point of both; hand-computed sequences."""
    seq = [[2.0, 1.0], [4.0, 3.0], [6.0, 9.0]]
    for est in (("ema", 1.0), ("history", 1)):
        st = {}
        for c in seq:
            assert S.smooth_cp(est, c, st) == c
    for est in (("ema", 0.3), ("history", 4)):
        st = {}
        for _ in range(6):
            np.testing.assert_allclose(S.smooth_cp(est, [1.5, 0.25], st), [1.5, 0.25], rtol=4e-16)
    st = {}
    out = [S.smooth_cp(("ema", 0.5), c, st) for c in seq]
    assert out == [[2.0, 1.0], [3.0, 2.0], [4.5, 5.5]]
    st = {}
    out = [S.smooth_cp(("history", 2), c, st) for c in seq]
    assert out == [[2.0, 1.0], [3.0, 2.0], [5.0, 6.0]]
    with pytest.raises(ValueError):
        S.smooth_cp(("median", 3), [1.0], {})


def _zero_grad(theta, x, y):
    return 0.0, np.zeros_like(theta)


def test_run_additive_delay_reaches_equal_times():
    """Model clock with speeds 1 and a delay of 4 on worker 1: X_m = n_m + d_m.
    From the even split [4, 4], Algorithm 1 moves to [5, 3], then [6, 2], where
    both workers take 6 (Eq. (3): equal predicted times) and it stays."""
    theta = np.zeros(2)
    batches = [(np.zeros((8, 2)), np.zeros(8, dtype=np.int64))] * 5
    out = S.run(_zero_grad, theta, batches, [[1.0, 1.0]] * 5, 1, 0.1, 0.0, 0.0, delays=[0.0, 4.0])
    assert out["partitions"] == [[4, 4], [5, 3], [6, 2], [6, 2], [6, 2]]
    assert out["xs"][0] == [4.0, 8.0] and out["xs"][2] == [6.0, 6.0]
    # window 0: the partition never moves (Sync-SGD); the slowest worker sets the step
    fixed = S.run(_zero_grad, theta, batches, [[1.0, 1.0]] * 5, 0, 0.1, 0.0, 0.0, delays=[0.0, 4.0])
    assert fixed["partitions"] == [[4, 4]] * 5 and fixed["cps"] == []
    assert [max(x) for x in fixed["xs"]] == [8.0] * 5


def test_run_cosine_schedule_closed_form():
    """With zero gradients and no momentum, theta_{t+1} = theta_t (1 - lr_t wd)."""
    theta = np.array([1.0, -2.0])
    T, wd = 6, 0.5
    batches = [(np.zeros((4, 2)), np.zeros(4, dtype=np.int64))] * T
    out = S.run(_zero_grad, theta, batches, [[1.0, 1.0]] * T, 2, 0.4, 0.0, wd, lr_total=T,
                lr_min=0.1)
    expect = theta.copy()
    for t in range(T):
        expect = expect * (1.0 - (0.1 + 0.3 * (1 + math.cos(math.pi * t / T)) / 2) * wd)
    np.testing.assert_allclose(out["theta"], expect, rtol=1e-15, atol=0)
