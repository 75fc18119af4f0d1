"""Oracle-side drivers of a synthetic workload: the workload's delay model and
mixing kind as oracle objects, column windows of its seeded inputs, and the
oracle's own evolution of those columns over several iterations.

TEST INFRASTRUCTURE (like the rest of ``oracle``): used by the test suite and
the benchmark's CPU-baseline leg only.  The workload description (``synth.workloads``)
is plain data; every name in it is mapped here to the oracle's own constants,
and the inputs are regenerated from ``synth`` (the seeded generator shared with
the GPU side, which holds none of the method's arithmetic).
"""

from __future__ import annotations

import numpy as np

from . import mixing, schedule, step

DELAY_KINDS = {"const": schedule.DELAY_CONST, "exp": schedule.DELAY_EXP,
               "lomax": schedule.DELAY_LOMAX}
ORDERS = {"mix_then_step": step.MIX_THEN_STEP, "step_then_mix": step.STEP_THEN_MIX}


def delay(wl) -> schedule.Delay:
    """The workload's delay model as the oracle's ``schedule.Delay``."""
    d = wl.delay
    return schedule.Delay(DELAY_KINDS[d.kind], d.base, d.param, d.slow_learner, d.slow_factor,
                          d.slow_prob)


def order(wl) -> int:
    return ORDERS[wl.order]


class Mixer:
    """W of every iteration for a mixing kind (Alg. 2 averaging step):
    ``uniform`` (ring all-reduce, Eq. 4-5), ``ring`` (D-PSGD, Eq. 6) or
    ``matcha`` (random matchings of a ``degree``-regular base graph, Sec. 6.1;
    MATCHA's optimised p and alpha when ``budget`` is set).  W is returned as
    the C ABI stores it, rounded to fp32, then widened back to fp64."""

    def __init__(self, kind: str, n: int, seed: int, degree: int = 3, budget=None):
        self.kind, self.n = kind, n
        self.matcha = None
        if kind == "matcha":
            self.matcha = mixing.Matcha(seed, n, degree)
            if budget is not None:
                self.matcha.optimize(budget)
        elif kind not in ("uniform", "ring"):
            raise ValueError(f"unknown mixing kind {kind}")

    def w(self, k: int) -> np.ndarray:
        if self.kind == "uniform":
            W = mixing.w_uniform(self.n)
        elif self.kind == "ring":
            W = mixing.w_ring(self.n)
        else:
            W = self.matcha.w(k)
        return W.astype(np.float32).astype(np.float64)


def mixer(wl) -> Mixer:
    return Mixer(wl.mixing, wl.n, wl.seed, wl.matcha_degree, wl.matcha_budget)


def window_inputs(wl, cols):
    """X0[n, len(cols)] and G[n, m, len(cols)] of a step workload at the given
    columns, regenerated on the host from the seeded input generator (flat
    index row * P + column of the contiguous [n, P] and [n, m, P] tensors)."""
    import synth
    from synth import workloads

    n, m, P = wl.n, wl.m, wl.P
    cols = np.asarray(cols, dtype=np.int64)
    xi = (np.arange(n, dtype=np.int64)[:, None] * P + cols[None, :]).reshape(-1)
    gi = (np.arange(n * m, dtype=np.int64)[:, None] * P + cols[None, :]).reshape(-1)
    X0 = synth.normal_f32(wl.seed, workloads.STREAM_X, xi, wl.x_std).reshape(n, len(cols))
    G = synth.normal_f32(wl.seed, workloads.STREAM_G, gi, wl.g_std).reshape(n, m, len(cols))
    return X0, G


def run(wl, X0, G, steps: int, first: int = 0, stop=None):
    """Evolves (X, V) with the oracle for iterations first .. first+steps-1 on
    fixed per-mini-batch gradients G (the step workloads keep G resident);
    returns X, V (fp64) and the list of per-iteration masks.  ``stop``
    (optional) is called after each iteration with its index and ends the run
    early when it returns True."""
    n, m = wl.n, wl.m
    X = np.asarray(X0, dtype=np.float64)
    V = np.zeros_like(X)
    mx, d, o = mixer(wl), delay(wl), order(wl)
    lr, mu = float(np.float32(wl.lr)), float(np.float32(wl.momentum))
    masks = []
    for k in range(first, first + steps):
        s = schedule.sample_schedule(wl.seed, k, n, m, d)
        masks.append(s["mask"])
        X, V = step.step(X, V, G, s["mask"], mx.w(k), lr, mu, o)
        if stop is not None and stop(k):
            break
    return X, V, masks
