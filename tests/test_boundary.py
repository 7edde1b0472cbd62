"""The C-ABI library on the host (no GPU needed): it loads, exports every
symbol include/*.h declares (hs.h, the step; hs_testing.h, measurement and tests), and its host-side parts (parameter layout,
compute-power estimate, repartition, Dynamic Partitioning window) agree with
the oracle exactly."""
import math
import os
import re

import numpy as np
import pytest

from oracle import models as Mo
from oracle import step as S

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

hs = pytest.importorskip("paper_2110_08941_amd.hs", reason="libhs.so not built")


def declared_symbols():
    text = "".join(open(os.path.join(ROOT, "include", f)).read()
                   for f in sorted(os.listdir(os.path.join(ROOT, "include"))) if f.endswith(".h"))
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(hs_[a-z0-9_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    names = declared_symbols()
    assert len(names) >= 20
    lib = hs.lib()
    for name in names:
        assert hasattr(lib, name), name
    assert set(names) == set(hs.EXPORTED)


@pytest.mark.parametrize("arch", ["mlp", "small_cnn", "resnet18", "resnet50", "vgg16"])
def test_param_layout_matches_oracle(arch):
    for dtype in ("fp32", "bf16"):
        m = hs.model_create(arch, dtype)
        try:
            net = Mo.build(arch)
            otab, oP = Mo.param_table(net)
            assert hs.num_params(m) == oP
            assert hs.num_true_params(m) == Mo.true_param_count(net)
            assert hs.param_table(m) == otab
            shape = (784,) if arch == "mlp" else (3, 32, 32)
            assert hs.forward_macs(m) == Mo.forward_flops(net, shape)
            assert hs.input_numel(m) == int(np.prod(shape))
        finally:
            hs.model_destroy(m)


def test_repartition_golden_and_random_bit_exact():
    from tests.test_oracle_step import load_cases
    for cp, total, expected in load_cases():
        assert hs.repartition(cp, total) == expected
    rng = np.random.default_rng(17)
    for _ in range(2000):
        m = int(rng.integers(1, 17))
        total = int(rng.integers(m, 10000))
        cp = [float(v) for v in np.exp(rng.normal(0, 1.0, size=m))]
        if rng.random() < 0.2:                          # exact ties
            cp = [float(rng.integers(1, 4)) for _ in range(m)]
        if rng.random() < 0.1:                          # shares that round to zero
            cp[0] = 1e-9
        assert hs.repartition(cp, total) == S.repartition(cp, total)


def test_estimate_cp_matches_oracle():
    rng = np.random.default_rng(3)
    for _ in range(200):
        m = int(rng.integers(1, 12))
        n = [int(v) for v in rng.integers(1, 500, size=m)]
        x = [float(v) for v in rng.uniform(1e-4, 3.0, size=m)]
        assert hs.estimate_cp(n, x) == S.estimate_cp(n, x)


def test_partitioner_matches_oracle_driver_logic():
    """The window logic of hs_partitioner_* against the oracle's driver, on
    random time traces: every partition bit-exact."""
    rng = np.random.default_rng(23)
    for trial in range(30):
        m = int(rng.integers(2, 9))
        total = int(rng.integers(4 * m, 3000))
        window = int(rng.integers(1, 6))
        steps = 4 * window + int(rng.integers(0, window))
        p = hs.Partitioner(m, total, window)
        n = S.even_split(m, total)
        xsum = [0.0] * m
        assert p.partition() == n
        for t in range(steps):
            tau = [float(v) for v in rng.uniform(0.5, 5.0, size=m)]
            speed = [float(v) for v in rng.uniform(0.5, 4.0, size=m)]
            cp = p.observe(p.partition(), tau, speed)
            for j in range(m):
                xsum[j] = xsum[j] + tau[j] / speed[j]
            if (t + 1) % window == 0:
                ocp = S.estimate_cp(n, [v / float(window) for v in xsum])
                assert cp == ocp
                n = S.repartition(ocp, total)
                xsum = [0.0] * m
            else:
                assert cp is None
            assert p.partition() == n
        p.close()


@pytest.mark.parametrize("est", [("ema", 0.5), ("ema", 0.37), ("history", 1), ("history", 3),
                                 ("history", 7)])
def test_partitioner_estimators_match_oracle(est):
    """hs_partitioner_set_estimator: EMA and history smoothing of the compute
    power across windows, against the oracle's smooth_cp on random traces;
    every estimate and partition bit-exact."""
    rng = np.random.default_rng(29)
    for trial in range(12):
        m = int(rng.integers(2, 9))
        total = int(rng.integers(4 * m, 3000))
        window = int(rng.integers(1, 4))
        p = hs.Partitioner(m, total, window)
        p.set_estimator(est[0], alpha=est[1] if est[0] == "ema" else 1.0,
                        history=est[1] if est[0] == "history" else 1)
        n, xsum, state = S.even_split(m, total), [0.0] * m, {}
        for t in range(10 * window):
            tau = [float(v) for v in rng.uniform(0.5, 5.0, size=m)]
            speed = [float(v) for v in rng.uniform(0.5, 4.0, size=m)]
            cp = p.observe(p.partition(), tau, speed)
            for j in range(m):
                xsum[j] = xsum[j] + tau[j] / speed[j]
            if (t + 1) % window == 0:
                ocp = S.smooth_cp(est, S.estimate_cp(n, [v / float(window) for v in xsum]), state)
                assert cp == ocp
                n = S.repartition(ocp, total)
                xsum = [0.0] * m
            assert p.partition() == n
        p.close()


def test_estimator_errors_and_reset():
    p = hs.Partitioner(3, 30, 1)
    for kind, alpha, hist in (("ema", 0.0, 1), ("ema", 1.5, 1), ("ema", float("nan"), 1),
                              ("history", 1.0, 0), ("history", 1.0, 5000)):
        with pytest.raises(hs.HSError):
            p.set_estimator(kind, alpha=alpha, history=hist)
    assert hs.lib().hs_partitioner_set_estimator(p.h, 9, 1.0, 1) == hs.HS_ERR_INVALID
    # switching estimators clears the carried state: history 2 after a reset
    # equals history 2 from scratch
    p.set_estimator("history", history=2)
    p.observe(p.partition(), [1.0, 2.0, 3.0], [1.0, 1.0, 1.0])
    p.set_estimator("history", history=2)
    q = hs.Partitioner(3, 30, 1)
    q.set_partition(p.partition())
    q.set_estimator("history", history=2)
    for _ in range(3):
        a = p.observe(p.partition(), [1.0, 2.0, 3.0], [1.0, 1.0, 1.0])
        b = q.observe(q.partition(), [1.0, 2.0, 3.0], [1.0, 1.0, 1.0])
        assert a == b
    p.close()
    q.close()


def test_model_clock_reaches_speed_proportional_partition():
    """Algorithm 1 with the model clock (X_m = n_m / s_m): even first window,
    then partitions proportional to the speeds (1:1:2:4 over 512 -> 64 64 128 256)."""
    p = hs.Partitioner(4, 512, 5)
    speeds = [1.0, 1.0, 2.0, 4.0]
    seen = []
    for t in range(20):
        n = p.partition()
        seen.append(n)
        p.observe(n, [float(v) for v in n], speeds)
    assert seen[0] == [128] * 4 and seen[4] == [128] * 4
    assert all(s == [64, 64, 128, 256] for s in seen[5:])


def test_error_paths():
    with pytest.raises(hs.HSError) as e:
        hs.repartition([1.0, float("nan")], 8)
    assert e.value.status == hs.HS_ERR_INVALID
    for bad in ([1.0, 0.0], [1.0, -2.0], [float("inf"), 1.0]):
        with pytest.raises(hs.HSError):
            hs.repartition(bad, 8)
    with pytest.raises(hs.HSError):
        hs.repartition([1.0, 1.0, 1.0], 2)
    with pytest.raises(hs.HSError):
        hs.estimate_cp([0, 3], [1.0, 1.0])
    with pytest.raises(hs.HSError):
        hs.model_create(7, "fp32")
    with pytest.raises(hs.HSError):
        hs.Partitioner(4, 3, 1)
    p = hs.Partitioner(2, 10, 1)
    with pytest.raises(hs.HSError):
        p.observe([5, 5], [1.0, float("nan")], [1.0, 1.0])
    with pytest.raises(hs.HSError):              # a step of another partition
        p.observe([4, 6], [1.0, 1.0], [1.0, 1.0])
    with pytest.raises(hs.HSError):
        p.set_partition([5, 4])
    assert p.partition() == [5, 5]                 # untouched by the failed calls
    m = hs.model_create("mlp", "fp32")
    with pytest.raises(hs.HSError):
        hs.workspace_create(m, 0)
    # argument errors are caught before any device work
    with pytest.raises(hs.HSError):
        hs.worker_grad(m, 0, 16, 0, 16, 16, 4, 16)
    with pytest.raises(hs.HSError):
        hs.weighted_average([16, 32], [0, 0], 64, 48)
    with pytest.raises(hs.HSError):
        hs.sgd_step(16, 32, 0, 64, 0.1, 0.9, 0.0)         # mu != 0 needs a momentum buffer
    with pytest.raises(hs.HSError):
        hs.wavg_sgd([16 + 4], [1], 64, 0, 64, 0.1, 0.0, 0.0)  # misaligned gradient
    for args in ((0, 4096, 64), (4096, 8192, 40), (4096, 4100, 64), (4096, 4096 + 32, 64)):
        with pytest.raises(hs.HSError):           # null, ragged, misaligned, overlapping
            hs.probe_copy(*args)
    for blocks, iters in ((0, 1), (1, 0), (65537, 1), (1, (1 << 20) + 1)):
        with pytest.raises(hs.HSError):
            hs.probe_mfma_loop(blocks, iters, 4096)
    with pytest.raises(hs.HSError):
        hs.probe_mfma_loop(1, 1, 0)
    hs.model_destroy(m)


def test_observation_of_another_partition_is_rejected():
    """An observation must describe a step run with the current partition: one
    launched before the window's repartition was observed is refused, and the
    state is unchanged (the next valid observation closes the window as if the
    refused one never came)."""
    p = hs.Partitioner(2, 12, 2)
    q = hs.Partitioner(2, 12, 2)
    for part in (p, q):
        part.observe([6, 6], [6.0, 6.0], [1.0, 3.0])
        assert part.observe([6, 6], [6.0, 6.0], [1.0, 3.0]) is not None
    assert p.partition() == [3, 9]
    with pytest.raises(hs.HSError):
        p.observe([6, 6], [6.0, 6.0], [1.0, 3.0])
    assert p.partition() == [3, 9]
    for part in (p, q):
        part.observe([3, 9], [3.0, 9.0], [1.0, 3.0])
        assert part.observe([3, 9], [3.0, 9.0], [1.0, 3.0]) is not None
    assert p.partition() == q.partition() == [3, 9]
    p.close()
    q.close()
