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
