"""Workload definitions: network, precision, total batch, workers, speeds,
repartition schedule and optimiser settings.

The paper's own runs (Section 5) use 128 samples per worker, momentum 0.9 and
weight decay 5e-4 on CIFAR10 with ResNet50/VGG16; the workloads below are
CIFAR-shaped MLP / small CNN / ResNet-18 / VGG-16 steps with simulated worker
speeds, sized for one GPU.
"""
from dataclasses import dataclass, field
from typing import Optional, Tuple


@dataclass(frozen=True)
class Workload:
    name: str
    arch: str                 # "mlp" | "small_cnn" | "resnet18" | "resnet50" | "vgg16"
    dtype: str                # "fp32" | "bf16"
    total: int                # N, samples per step over all workers
    speeds: Tuple[float, ...] # initial simulated speed s_m of every worker
    steps: int                # steps of the workload
    window: int               # repartition every `window` steps (0: never)
    start_even: bool          # first window uses the even split (Algorithm 1)
    drift_sigma: float        # multiplicative random-walk sigma of the speeds
    lr: float
    mu: float
    wd: float

    @property
    def workers(self):
        return len(self.speeds)

    @property
    def in_shape(self):
        return (784,) if self.arch == "mlp" else (3, 32, 32)


WORKLOADS = {
    # MLP 784-256-10, fp32, N=256 over 2 workers of speed 1:3, one plain SGD step.
    "mlp_fp32": Workload("mlp_fp32", "mlp", "fp32", 256, (1.0, 3.0), 1, 0, False, 0.0,
                         0.1, 0.0, 0.0),
    # Small CNN, fp32, N=512 over 4 workers 1:1:2:4, 20 steps, repartition every 5.
    "smallcnn_fp32": Workload("smallcnn_fp32", "small_cnn", "fp32", 512, (1.0, 1.0, 2.0, 4.0),
                              20, 5, True, 0.0, 0.1, 0.0, 0.0),
    # ResNet-18 (CIFAR), fp32, N=1024 over 4 workers 1:1.5:2:3.5, momentum SGD.
    "resnet18_fp32": Workload("resnet18_fp32", "resnet18", "fp32", 1024, (1.0, 1.5, 2.0, 3.5),
                              1, 0, False, 0.0, 0.1, 0.9, 5e-4),
    # ResNet-18 (CIFAR), bf16 operands / fp32 master, N=2048 over 8 drifting
    # workers, repartition every 10 steps over 100 steps.
    "resnet18_bf16": Workload("resnet18_bf16", "resnet18", "bf16", 2048,
                              (1.0, 1.0, 1.0, 2.0, 2.0, 4.0, 4.0, 8.0), 100, 10, True, 0.05,
                              0.1, 0.9, 5e-4),
    # ResNet-50 (CIFAR, bottleneck blocks), bf16 operands / fp32 master,
    # N=1024 (128 per worker, as in Section 5) over 8 drifting workers,
    # repartition every 10 steps over 100 steps.
    "resnet50_bf16": Workload("resnet50_bf16", "resnet50", "bf16", 1024,
                              (1.0, 1.0, 1.0, 2.0, 2.0, 4.0, 4.0, 8.0), 100, 10, True, 0.05,
                              0.1, 0.9, 5e-4),
    # VGG-16 (CIFAR), bf16, N=4096 over 8 workers 1:1:1:2:2:4:4:8.
    "vgg16_bf16": Workload("vgg16_bf16", "vgg16", "bf16", 4096,
                           (1.0, 1.0, 1.0, 2.0, 2.0, 4.0, 4.0, 8.0), 1, 0, False, 0.0,
                           0.1, 0.9, 5e-4),
}

# Standalone weighted-average + SGD: 8 fp32 gradient buffers of 25M elements,
# partition sizes of the VGG-16 workload.
STANDALONE_WAVG = {"workers": 8, "numel": 25_000_000,
                   "n": (178, 178, 178, 356, 356, 713, 712, 1425), "lr": 0.1}
