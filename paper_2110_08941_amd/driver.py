"""Multi-step driver of the heterogeneous data-parallel step on one GPU.

Each step (all device work through libhs):
  * worker m gets rows [o_m, o_m + n_m) of the step's batch and runs
    hs_worker_grad on its own HIP stream, bracketed by timing events;
  * the main stream waits for every worker, then hs_wavg_sgd forms the
    partition-weighted gradient and applies the SGD step in one pass;
  * the workers' times tau_m feed the Dynamic Partitioning state
    (hs_partitioner_observe), which divides them by the simulated speeds
    s_m, and at the end of every window repartitions the batch in proportion
    to the estimated compute powers (Eq. (2), Algorithm 1).
With clock="model" the time of worker m is n_m (X_m = n_m / s_m), which
makes the partition sequence independent of the hardware.

grouped=True runs all workers in one hs_workers_grad call on the main stream
(every layer launched once over the whole batch, statistics, losses and
weight gradients per worker).  Per-worker device times do not exist there,
so it requires clock="model".
PyTorch is used for device memory, streams and events only.
"""
import math

import numpy as np
import torch

from . import hs, synth
from .configs import WORKLOADS, Workload


class Trainer:
    def __init__(self, workload, seed=0, clock="measured", device="cuda:0", n_batches=4,
                 max_n=None, steps=None, theta0=None, grouped=False, exchange="edp",
                 delays=None, estimator=("window",), lr_schedule=None, serial=False,
                 fused_avg=False):
        self.wl = wl = WORKLOADS[workload] if isinstance(workload, str) else workload
        assert isinstance(wl, Workload)
        if clock not in ("measured", "model"):
            raise ValueError("clock must be 'measured' or 'model'")
        if grouped and serial:
            raise ValueError("serial applies to per-worker launches, not grouped ones")
        if grouped and clock != "model":
            raise ValueError("grouped workers have no per-worker device time: use clock='model'")
        if fused_avg and (not grouped or exchange != "edp"):
            raise ValueError("fused_avg needs grouped workers and the edp exchange")
        if exchange not in ("edp", "mean"):
            raise ValueError("exchange must be 'edp' or 'mean'")
        if estimator[0] not in ("window", "ema", "history"):
            raise ValueError("unknown estimator %r" % (estimator,))
        if lr_schedule is not None and (lr_schedule[0] != "cosine" or lr_schedule[1] <= 0):
            raise ValueError("lr_schedule must be None or ('cosine', total_steps > 0, lr_min)")
        if delays is not None and (len(delays) != wl.workers or
                                   not all(math.isfinite(d) and d >= 0.0 for d in delays)):
            raise ValueError("delays: one finite, non-negative delay per worker")
        self.clock = clock
        self.grouped = grouped
        # fused_avg: the one-pass call forms the partition-weighted gradient
        # itself (hs_workers_grad_wavg) and the step applies plain SGD to it
        self.fused_avg = fused_avg
        # exchange: "edp" weights g_m by n_m / N (Section 4.2); "mean" is the
        # plain mean of Sync-SGD and DP-SGD.  delays: additive per-batch delay
        # of each worker in the units of X (Section 5's simulated
        # heterogeneity).  estimator: compute power across windows, ("window",),
        # ("ema", alpha) or ("history", h).  lr_schedule: None (constant) or
        # ("cosine", total_steps, lr_min).  serial: the workers run one after
        # another on one stream (sharing one workspace), so that each worker's
        # measured time is its own work alone, as on a device of its own.
        self.exchange = exchange
        self.delays = None if delays is None else [float(d) for d in delays]
        self.lr_schedule = lr_schedule
        self.dev = torch.device(device)
        self.M, self.N = wl.workers, wl.total
        # the Dynamic Partitioning state first: its argument errors leave
        # nothing allocated
        self.part = hs.Partitioner(self.M, self.N, wl.window)
        try:
            if estimator[0] == "ema":
                self.part.set_estimator("ema", alpha=estimator[1])
            elif estimator[0] == "history":
                self.part.set_estimator("history", history=estimator[1])
        except Exception:
            self.part.close()
            raise
        self.steps = steps if steps is not None else wl.steps
        self.model = hs.model_create(wl.arch, wl.dtype)
        self.P = hs.num_params(self.model)
        self.table = hs.param_table(self.model)
        self.bf16 = wl.dtype == "bf16"
        th = synth.he_normal(self.table, self.P, seed) if theta0 is None else theta0
        self.theta = torch.tensor(np.asarray(th, dtype=np.float32), device=self.dev)
        self.theta_bf16 = torch.empty(self.P, dtype=torch.int16, device=self.dev) if self.bf16 else None
        if self.bf16:
            hs.params_to_bf16(self.theta.data_ptr(), self.theta_bf16.data_ptr(), self.P)
        self.mom = torch.zeros(self.P, device=self.dev) if wl.mu != 0.0 else None
        self.grads = [torch.empty(self.P, device=self.dev)
                      for _ in range(1 if fused_avg else self.M)]
        self.losses = torch.zeros(self.M, device=self.dev)
        self.max_n = max_n or self.N
        if grouped:
            self.streams = []
            self.ws = [hs.workspace_create(self.model, self.N)]
        elif serial:
            self.streams = [torch.cuda.Stream(device=self.dev)] * self.M
            self.ws = [hs.workspace_create(self.model, self.max_n)]
        else:
            self.streams = [torch.cuda.Stream(device=self.dev) for _ in range(self.M)]
            self.ws = [hs.workspace_create(self.model, self.max_n) for _ in range(self.M)]
        if not wl.start_even:                       # fixed split in proportion to the speeds
            self.part.set_partition(hs.repartition(list(wl.speeds), self.N))
        self.speeds = synth.speed_schedule(wl.speeds, max(self.steps, 1), seed, wl.drift_sigma)
        self.in_numel = hs.input_numel(self.model)
        self.batches = []
        for b in range(n_batches):
            x, y = synth.batch(wl.in_shape, self.N, seed, b)
            self.batches.append((torch.from_numpy(x).to(self.dev), torch.from_numpy(y).to(self.dev)))
        self.t = 0
        self.in_window = 0      # steps launched since the current window started
        self.time_opt = False   # record events around the weighted-average + SGD launch
        self.opt_events = []
        self.pending = []       # (step, partition, [(e0, e1)] or None) awaiting observation
        self.log = []           # per step: partition, tau, cp (if a window closed)

    # ------------------------------------------------------------------ step
    def batch(self, t):
        return self.batches[t % len(self.batches)]

    def launch_workers(self, n, x, y, timed=True):
        """Worker gradients on their streams; the main stream waits for all."""
        main = torch.cuda.current_stream(self.dev)
        ready = torch.cuda.Event()
        ready.record(main)
        events, o = [], 0
        ew = x.element_size() * self.in_numel
        for m in range(self.M):
            s = self.streams[m]
            s.wait_event(ready)
            e0 = e1 = None
            if timed:
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record(s)
            hs.worker_grad(self.model, self.ws[m % len(self.ws)], self.theta.data_ptr(),
                           self.theta_bf16.data_ptr() if self.bf16 else 0,
                           x.data_ptr() + o * ew, y.data_ptr() + o * 4, n[m],
                           self.grads[m].data_ptr(), self.losses.data_ptr() + 4 * m,
                           s.cuda_stream)
            if timed:
                e1.record(s)
            else:
                e1 = torch.cuda.Event()
                e1.record(s)
            events.append((e0, e1))
            o += n[m]
        for _, e1 in events:
            main.wait_event(e1)
        return events

    def step(self):
        """One synchronous step; returns the partition it used."""
        wl, t = self.wl, self.t
        n = self.part.partition()
        x, y = self.batch(t)
        main = torch.cuda.current_stream(self.dev)
        if self.fused_avg:
            hs.workers_grad_wavg(self.model, self.ws[0], self.theta.data_ptr(),
                                 self.theta_bf16.data_ptr() if self.bf16 else 0, x.data_ptr(),
                                 y.data_ptr(), n, self.grads[0].data_ptr(),
                                 self.losses.data_ptr(), main.cuda_stream)
            events = None
        elif self.grouped:
            hs.workers_grad(self.model, self.ws[0], self.theta.data_ptr(),
                            self.theta_bf16.data_ptr() if self.bf16 else 0, x.data_ptr(),
                            y.data_ptr(), n, [g.data_ptr() for g in self.grads],
                            self.losses.data_ptr(), main.cuda_stream)
            events = None
        else:
            events = self.launch_workers(n, x, y, timed=(self.clock == "measured"))
        if self.time_opt:
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(main)
        # the kernel weights worker m by w[m] / sum w: the partition sizes, or
        # ones for the plain mean
        if self.fused_avg:
            hs.sgd_step(self.theta.data_ptr(), self.grads[0].data_ptr(),
                        self.mom.data_ptr() if self.mom is not None else 0, self.P, self.lr(t),
                        wl.mu, wl.wd, self.theta_bf16.data_ptr() if self.bf16 else 0,
                        main.cuda_stream)
        else:
            w = n if self.exchange == "edp" else [1] * self.M
            hs.wavg_sgd([g.data_ptr() for g in self.grads], w, self.theta.data_ptr(),
                        self.mom.data_ptr() if self.mom is not None else 0, self.P, self.lr(t),
                        wl.mu, wl.wd, self.theta_bf16.data_ptr() if self.bf16 else 0,
                        main.cuda_stream)
        if self.time_opt:
            e1.record(main)
            self.opt_events.append((e0, e1))
        self.pending.append((t, n, events))
        self.t += 1
        # the last step of a window is observed before the next step reads
        # its partition, so that every observation of a window describes a
        # step run with that window's partition (a flush in between, e.g.
        # after warm-up steps, only observes steps earlier)
        self.in_window += 1
        if wl.window > 0 and self.in_window == wl.window:
            self.flush()
            self.in_window = 0
        elif len(self.pending) >= 64:
            self.flush()
        return n

    def lr(self, t):
        """Learning rate of step t: constant, or cosine annealing
        lr_min + (lr - lr_min) (1 + cos(pi t / total)) / 2."""
        if self.lr_schedule is None:
            return self.wl.lr
        _, total, lr_min = self.lr_schedule
        return lr_min + (self.wl.lr - lr_min) * (1.0 + math.cos(math.pi * t / total)) / 2.0

    def flush(self):
        """Report the pending steps' times to the partitioner, in step order.
        The batch time of worker m is X_m = tau_m / s_m (+ delay_m)."""
        for t, n, events in self.pending:
            if self.clock == "measured":
                for _, e1 in events:
                    e1.synchronize()
                tau = [float(e0.elapsed_time(e1)) for e0, e1 in events]
            else:
                tau = [float(v) for v in n]
            speed = self.speeds[min(t, len(self.speeds) - 1)]
            x = [tau[m] / float(speed[m]) for m in range(self.M)]
            if self.delays is not None:
                x = [x[m] + self.delays[m] for m in range(self.M)]
            cp = None
            if self.wl.window > 0:
                # with delays the batch times are reported whole (speed 1)
                cp = (self.part.observe(n, tau, speed) if self.delays is None
                      else self.part.observe(n, x, [1.0] * self.M))
            self.log.append({"step": t, "n": list(n), "tau": tau, "speed": list(speed), "x": x,
                             "xmax": max(x), "cp": cp})
        self.pending = []

    def opt_bytes(self):
        """Algorithmic HBM bytes of one weighted-average + SGD launch: M fp32
        gradients read (one, the weighted gradient, with fused_avg), theta
        read and written, the momentum buffer read and written (if any), the
        bf16 copy written (if any)."""
        b = (1 if self.fused_avg else self.M) * 4 + 8
        if self.mom is not None:
            b += 8
        if self.bf16:
            b += 2
        return b * self.P

    def run(self, steps=None):
        for _ in range(steps if steps is not None else self.steps):
            self.step()
        self.flush()

    def close(self):
        for w in self.ws:
            hs.workspace_destroy(w)
        self.ws = []
        self.part.close()
        hs.model_destroy(self.model)
        self.model = None
