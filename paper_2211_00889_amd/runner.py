"""Drives the hot path for a workload: device buffers resident in HBM, and per
iteration the simulated schedule and mixing matrix (host library calls) then
one fused ``nbsgd_step`` (gfx950 kernel) on the caller's stream.

The host work of iteration k+1 overlaps the kernel of iteration k because the
step launch is asynchronous and copies its per-step constants into the kernel
arguments.
"""

from __future__ import annotations

import numpy as np

from . import _lib
from ._lib import DELAY_CONST, DELAY_EXP, DELAY_LOMAX, MIX_THEN_STEP, STEP_THEN_MIX

_DELAY = {"const": DELAY_CONST, "exp": DELAY_EXP, "lomax": DELAY_LOMAX}
_ORDER = {"mix_then_step": MIX_THEN_STEP, "step_then_mix": STEP_THEN_MIX}


class Mixer:
    """Per-iteration mixing matrix of a workload's kind."""

    def __init__(self, kind: str, n: int, seed: int, degree: int = 3, budget=None):
        self.kind = kind
        self.matcha = None
        if kind == "uniform":
            self.fixed = _lib.w_allreduce(n)
        elif kind == "ring":
            self.fixed = _lib.w_ring(n)
        elif kind == "matcha":
            self.matcha = _lib.Matcha(seed, n, degree)
            if budget is not None:  # MATCHA's optimised probabilities and alpha
                self.matcha.optimize(budget)
        else:
            raise ValueError(f"unknown mixing kind {kind}")

    def w(self, step: int) -> np.ndarray:
        if self.matcha is not None:
            return self.matcha.w(step)[0]
        return self.fixed


class Schedule:
    """Finished-mini-batch mask of each iteration for a workload's delay model."""

    def __init__(self, wl):
        d = wl.delay
        self.args = (wl.n, wl.m, _DELAY[d.kind], d.base, d.param, d.slow_learner, d.slow_factor,
                     d.slow_prob)
        self.seed = wl.seed

    def mask(self, step: int):
        n, m, kind, base, param, slow, factor, prob = self.args
        return _lib.sample_mask(self.seed, step, n, m, kind, base, param, slow, factor, prob)


class StepRunner:
    """Replicas X, momentum V and gradients G of one workload on a device.

    Rows are allocated ``ld = nbsgd_row_stride(P)`` floats apart (P itself
    up to 2^20, the next power of two up to 2^22, else a multiple of 2^22 so
    rows start on 16 MiB boundaries);
    ``X``, ``V`` and ``G`` are the [.., P] views of the parameters.  Every row
    holds the values the generator gives the contiguous [n, P] / [n, m, P]
    tensor (flat index row * P + column)."""

    def __init__(self, wl, device="cuda:0", P: int | None = None, fill: bool = True):
        import torch

        from synth import device as synth_device
        from synth import workloads

        self.wl = wl
        self.P = wl.P if P is None else P
        n, m, P = wl.n, wl.m, self.P
        self.ld = _lib.row_stride(P)
        self.device = torch.device(device)
        self.Xrows = torch.empty((n, self.ld), dtype=torch.float32, device=self.device)
        self.Vrows = torch.zeros((n, self.ld), dtype=torch.float32, device=self.device)
        self.Grows = torch.empty((n, m, self.ld), dtype=torch.float32, device=self.device)
        self.X, self.V, self.G = self.Xrows[:, :P], self.Vrows[:, :P], self.Grows[:, :, :P]
        if fill:
            for i in range(n):
                synth_device.fill_normal(self.Xrows[i, :P], wl.seed, workloads.STREAM_X, wl.x_std,
                                         first=i * P)
                for j in range(m):
                    synth_device.fill_normal(self.Grows[i, j, :P], wl.seed, workloads.STREAM_G,
                                             wl.g_std, first=(i * m + j) * P)
        self.order = _ORDER[wl.order]
        self.mixer = Mixer(wl.mixing, n, wl.seed, wl.matcha_degree, wl.matcha_budget)
        self.schedule = Schedule(wl)

    def plan(self, step: int):
        """Host half of iteration ``step``: (mask, counts, timing, W)."""
        mask, counts, _, timing = self.schedule.mask(step)
        return mask, counts, timing, self.mixer.w(step)

    def launch(self, mask, W, stream=None):
        _lib.step_strided(self.Xrows, self.Vrows, self.Grows, self.P, mask, W, self.wl.lr,
                          self.wl.momentum, self.order, stream)

    def run(self, steps: int, first: int = 0, stream=None):
        """Runs iterations first .. first+steps-1; returns the per-step counts."""
        out = []
        for k in range(first, first + steps):
            mask, counts, _, W = self.plan(k)
            self.launch(mask, W, stream)
            out.append(counts)
        return out


class MlpRunner:
    """The end-to-end workload on a device: synthetic data and labels, n
    identical initial replicas, and per iteration the schedule, the shuffled
    mini-batch indices, the per-mini-batch gradients (bf16 MFMA) and the fused
    step with the workload's mixing kind (ring, MATCHA or uniform W)."""

    def __init__(self, wl, device="cuda:0", data=None, labels=None, x0=None):
        import torch

        from synth import mlp_data

        self.wl = wl
        self.dims = (wl.d_in, wl.hidden, wl.classes)
        self.P = _lib.mlp_param_count(*self.dims)
        dev = self.device = torch.device(device)
        if data is None:
            data = mlp_data.inputs(wl.seed, wl.n_samples, wl.d_in)
        if labels is None:
            labels = mlp_data.teacher_labels(wl.seed, data, wl.hidden, wl.classes)
        if x0 is None:
            x0 = mlp_data.student_init(wl.seed, wl.d_in, wl.hidden, wl.classes)
        self.data = torch.from_numpy(np.ascontiguousarray(data, dtype=np.float32)).to(dev)
        self.labels = torch.from_numpy(np.ascontiguousarray(labels, dtype=np.int32)).to(dev)
        x0 = np.asarray(x0, dtype=np.float32)
        row = np.zeros(self.P, np.float32)  # the library's layout pads the vector with zeros
        row[:x0.size] = x0
        # rows ld floats apart (the fused step's row stride); X, V, G view the
        # first P columns
        P, ld = self.P, _lib.row_stride(self.P)
        self.ld = ld
        self.Xrows = torch.zeros((wl.n, ld), dtype=torch.float32, device=dev)
        self.Xrows[:, :P] = torch.from_numpy(row).to(dev)
        self.Vrows = torch.zeros((wl.n, ld), dtype=torch.float32, device=dev)
        self.Grows = torch.zeros((wl.n, wl.m, ld), dtype=torch.float32, device=dev)
        self.X, self.V, self.G = self.Xrows[:, :P], self.Vrows[:, :P], self.Grows[:, :, :P]
        self.losses = torch.zeros(wl.n * wl.m, dtype=torch.float32, device=dev)
        self.eval_idx = wl.eval_indices()
        self.eval_losses = torch.zeros(len(self.eval_idx) // wl.batch, dtype=torch.float32, device=dev)
        rows = max(wl.n * wl.m * wl.batch, len(self.eval_idx))
        ws = _lib.mlp_workspace_bytes(*self.dims, rows)
        self.workspace = torch.empty((ws + 15) // 16 * 4, dtype=torch.float32, device=dev)
        self.mean = torch.zeros_like(self.Xrows)
        self.mixer = Mixer(wl.mixing, wl.n, wl.seed, wl.matcha_degree, wl.matcha_budget)
        self.schedule = Schedule(wl)
        self.last_schedule = None
        self.order = _ORDER[wl.order]
        self.w_mean = _lib.w_allreduce(wl.n)

    def step(self, k: int, stream=None, blocking: bool = False, events=None):
        """Iteration k; returns (mask, counts, seconds): the finished mask, the
        finished counts and the iteration's simulated wall time.  Non-blocking
        (Alg. 2): the schedule's mask, time T_step (the terminal signal, or a
        forced first mini-batch if later).  ``blocking``: the D-PSGD baseline
        on the same W, every learner finishes all m mini-batches and the
        iteration waits for the slowest, T_sync (the synchronous baseline of
        the workload's mixing kind: D-PSGD, MATCHA or all-reduce).  The
        finished mini-batches' losses are left in ``self.losses`` (index i*m +
        j).  ``events``: a list that receives three recorded device events
        (before the gradients, between gradients and step, after the step).
        The iteration's schedule (mask, counts, per-mini-batch times, timing)
        is kept in ``last_schedule``."""
        wl = self.wl
        mask, counts, times, timing = self.schedule.mask(k)
        self.last_schedule = (mask, counts, times, timing)
        seconds = float(timing[2])
        if blocking:
            mask = np.ones_like(mask)
            counts = np.full_like(counts, wl.m)
            seconds = float(timing[1])
        idx = _lib.minibatch_indices(wl.seed, k, wl.n, wl.m, wl.batch, wl.shard)
        W = self.mixer.w(k)
        ev = None
        if events is not None:
            import torch

            ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
            ev[0].record(stream)
        _lib.mlp_grad_strided(self.Xrows, wl.m, self.dims, self.data, self.labels, idx, mask,
                              self.Grows, self.losses, self.workspace, stream)
        if ev is not None:
            ev[1].record(stream)
        _lib.step_strided(self.Xrows, self.Vrows, self.Grows, self.P, mask, W, wl.lr, wl.momentum,
                          self.order, stream)
        if ev is not None:
            ev[2].record(stream)
            events.append(ev)
        return mask, counts, seconds

    def evaluate(self, stream=None):
        """Loss of the average replica (the method's output) on the fixed
        evaluation samples, per batch of 32 (device tensor)."""
        # whole rows: the padding columns hold zeros and average to zeros
        _lib.mix(self.Xrows, self.w_mean, self.mean, stream)
        _lib.mlp_loss(self.mean[0, :self.P], self.dims, self.data, self.labels, self.eval_idx, self.eval_losses,
                      self.workspace, stream)
        return self.eval_losses
