"""The multi-step driver rejects bad options before it allocates anything
(host only: no GPU needed)."""
import pytest

hs = pytest.importorskip("paper_2110_08941_amd.hs", reason="libhs.so not built")


@pytest.mark.parametrize("kw", [
    dict(exchange="median"),
    dict(estimator=("median", 3)),
    dict(lr_schedule=("step", 10, 0.0)),
    dict(lr_schedule=("cosine", 0, 0.0)),
    dict(delays=[1.0, 2.0]),                      # the workload has 4 workers
    dict(delays=[1.0, -1.0, 0.0, 0.0]),
    dict(delays=[float("nan"), 0.0, 0.0, 0.0]),
    dict(clock="wall"),
    dict(grouped=True, clock="measured"),
    dict(grouped=True, clock="model", serial=True),
])
def test_bad_options_raise_value_error(kw):
    from paper_2110_08941_amd.driver import Trainer
    with pytest.raises(ValueError):
        Trainer("smallcnn_fp32", **kw)


@pytest.mark.parametrize("est", [("ema", 0.0), ("ema", 1.5), ("history", 0), ("history", 2000)])
def test_bad_estimator_parameters_raise_from_the_library(est):
    from paper_2110_08941_amd.driver import Trainer
    with pytest.raises(hs.HSError):
        Trainer("smallcnn_fp32", estimator=est)
