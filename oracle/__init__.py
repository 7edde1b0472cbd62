"""CPU oracle for one heterogeneous data-parallel training step (test infrastructure).

This package is the plain, slow, obviously-correct definition that the GPU
library is checked against.  It is TEST INFRASTRUCTURE: only the test suite,
the smoke check and the CPU-baseline leg of the benchmark may import it.  The
product path (the C-ABI library and its Python binding) never imports, calls
or links anything here, and this package imports nothing from the product.

Everything is computed in float64 with numpy.  A library matmul is used as
one step of a convolution or linear layer (one matmul per kernel tap); there
is no other blocking, fusion or reordering.

What the step computes, and the passage of the paper each part follows
(arXiv 2110.08941, "Distributed Optimization using Heterogeneous Compute
Systems"):

* Per-worker gradient of the mean loss over the worker's partition --
  Section 1, Eq. (1) (f_m is the expectation over worker m's data) and the
  Sync-SGD description in the same section.            -> ``models``, ``layers``
* Partition-size-weighted gradient average (the Enhanced Dynamic Partitioning
  weighting by normalised compute power) -- Section 4.2.   -> ``step.weighted_average``
* SGD with momentum and weight decay -- Section 1 (update rule) and
  Section 5 (momentum 0.9, weight decay 5e-4).        -> ``step.sgd_step``
* Compute-power estimate CP_m = |D_m| / X_m -- Section 4, Eq. (2).
                                                       -> ``step.estimate_cp``
* Throughput-proportional repartition -- Section 4.1, Algorithm 1.
                                                       -> ``step.repartition``

Pins (tests that check this oracle against something other than itself) are
listed in ``tests/test_oracle_*.py``.  Parity unpinned: the size of the bf16
rounding error of the GPU path (only bounded by the stated tolerance) and the
measured per-worker times (hardware dependent; the repartition of any given
time vector is pinned, the times themselves are not).
"""
