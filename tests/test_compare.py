"""The Section 5 comparison report: host-side statistics on hand-made batch
times (CPU), and a small run of every mode on the GPU with the model clock,
whose step times have closed forms."""
import json

import numpy as np
import pytest

from paper_2110_08941_amd import compare as C
from tests.gpu_util import require_gpu


def test_delay_vector():
    assert C.delay_vector(4, [0, 1], 2.5) == [2.5, 2.5, 0.0, 0.0]
    assert C.delay_vector(3, [], 1.0) == [0.0, 0.0, 0.0]
    with pytest.raises(ValueError):
        C.delay_vector(2, [2], 1.0)


def test_summarize_hand_example():
    """Two workers over three steps: step time max_m X_m, each worker's wait
    for the slowest, histograms over shared edges."""
    xs = [[2.0, 4.0], [3.0, 3.0], [5.0, 1.0]]
    edges = [0.0, 2.0, 4.0, 6.0]
    s = C.summarize(xs, edges)
    assert s["steps"] == 3
    assert s["max_x_mean"] == 4.0 and s["max_x_max"] == 5.0 and s["sim_time"] == 12.0
    # step times 4, 3, 5: worker 0 waits 2, 0, 0; worker 1 waits 0, 0, 4
    assert s["x_mean"] == pytest.approx([10.0 / 3, 8.0 / 3], abs=1e-15)
    assert s["wait_mean"] == pytest.approx([2.0 / 3, 4.0 / 3], abs=1e-15)
    assert s["wait_frac"] == pytest.approx([2.0 / 12, 4.0 / 12], abs=1e-15)
    assert s["spread_mean"] == pytest.approx(2.0, abs=1e-15)
    # bins [0,2) [2,4) [4,6]: worker 0 has 2, 3, 5; worker 1 has 4, 3, 1
    assert s["hist"] == [[0, 2, 1], [1, 1, 1]]
    # skipping the first step
    s1 = C.summarize(xs, edges, skip=1)
    assert s1["steps"] == 2 and s1["max_x_mean"] == 4.0
    with pytest.raises(ValueError):
        C.summarize(xs, edges, skip=3)


def test_shared_edges_cover_all_runs():
    e = C.shared_edges([[[1.0, 2.0]], [[0.5, 7.0]]], 4)
    assert e[0] == 0.5 and e[-1] == 7.0 and len(e) == 5
    e = C.shared_edges([[[3.0, 3.0]]], 2)
    assert e[0] == 3.0 and e[-1] == 4.0


@pytest.mark.gpu
def test_compare_model_clock_closed_form(capsys):
    """Small CNN, N = 512 over 4 equal workers, delay 0.5 x 128 = 64 on workers
    0 and 1, model clock (X_m = n_m + delay_m), 20 steps, window 5.  Sync-SGD:
    X = 192, 192, 128, 128 every step.  Dynamic Partitioning moves the split
    through 102/154 and 97/159 to the fixed point 96, 96, 160, 160 of Eq. (3),
    where every X_m = 160; the window step times are 192, 166, 161, 160.  DP
    and EDP take the same partitions (the model clock does not see the
    exchange)."""
    require_gpu()
    rc = C.main(["--workload", "smallcnn_fp32", "--steps", "20", "--window", "5", "--clock",
                 "model", "--delay-frac", "0.5", "--modes", "sync,dp,edp"])
    assert rc == 0
    rep = json.loads(capsys.readouterr().out.strip().splitlines()[-1])
    assert rep["delay"] == 64.0 and rep["delayed"] == [0, 1] and rep["window"] == 5
    sync, dp, edp = (rep["modes"][k] for k in ("sync", "dp", "edp"))
    assert sync["x_mean"] == [192.0, 192.0, 128.0, 128.0] and sync["max_x_mean"] == 192.0
    assert sync["final_partition"] == [128] * 4
    assert dp["final_partition"] == [96, 96, 160, 160] == edp["final_partition"]
    assert dp["max_x_mean"] == (192.0 + 166.0 + 161.0 + 160.0) / 4 == edp["max_x_mean"]
    assert sync["wait_mean"] == [0.0, 0.0, 64.0, 64.0]
    assert dp["speedup_vs_sync"] == pytest.approx(192.0 / 169.75, rel=1e-15)
    for v in (sync, dp, edp):
        assert np.isfinite(v["loss_last"]) and v["loss_last"] < v["loss_first"] * 1.5
