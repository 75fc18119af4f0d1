"""Shared test helpers: the parity metric and oracle-side drivers."""

from __future__ import annotations

import numpy as np

import oracle
import synth
from synth import gen, workloads

# Parity bar for fp32 results: max_k |got_k - want_k| / max(|want_k|, rms(want))
# over each tensor (X and V separately).  Stated for the step in fp32 against
# the fp64 oracle; the max(|want|, rms) floor keeps near-zero elements from
# turning rounding noise into huge relative errors.
TOL = 1e-5

ORACLE_DELAY = {"const": oracle.schedule.DELAY_CONST, "exp": oracle.schedule.DELAY_EXP,
                "lomax": oracle.schedule.DELAY_LOMAX}
ORACLE_ORDER = {workloads.MIX_THEN_STEP: oracle.step.MIX_THEN_STEP,
                workloads.STEP_THEN_MIX: oracle.step.STEP_THEN_MIX}


def rel_err(got, want) -> float:
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    if want.size == 0:
        return 0.0
    rms = float(np.sqrt(np.mean(want * want)))
    denom = np.maximum(np.abs(want), rms if rms > 0 else 1.0)
    return float(np.max(np.abs(got - want) / denom))


def oracle_delay(wl):
    d = wl.delay
    return oracle.schedule.Delay(ORACLE_DELAY[d.kind], d.base, d.param, d.slow_learner, d.slow_factor,
                                 d.slow_prob)


class OracleMixer:
    def __init__(self, wl):
        self.wl = wl
        self.matcha = oracle.mixing.Matcha(wl.seed, wl.n, wl.matcha_degree) \
            if wl.mixing == "matcha" else None
        if self.matcha is not None and wl.matcha_budget is not None:
            self.matcha.optimize(wl.matcha_budget)

    def w(self, step):
        """The oracle's W, stored in the ABI's fp32 and widened back to fp64."""
        if self.wl.mixing == "uniform":
            W = oracle.mixing.w_uniform(self.wl.n)
        elif self.wl.mixing == "ring":
            W = oracle.mixing.w_ring(self.wl.n)
        else:
            W = self.matcha.w(step)
        return W.astype(np.float32).astype(np.float64)


def window_inputs(wl, cols):
    """X0[n, len(cols)] and G[n, m, len(cols)] of the workload at the given
    columns, regenerated on the host from the input generator."""
    n, m, P = wl.n, wl.m, wl.P
    cols = np.asarray(cols, dtype=np.int64)
    xi = (np.arange(n, dtype=np.int64)[:, None] * P + cols[None, :]).reshape(-1)
    gi = (np.arange(n * m, dtype=np.int64)[:, None] * P + cols[None, :]).reshape(-1)
    X0 = synth.normal_f32(wl.seed, workloads.STREAM_X, xi, wl.x_std).reshape(n, len(cols))
    G = synth.normal_f32(wl.seed, workloads.STREAM_G, gi, wl.g_std).reshape(n, m, len(cols))
    return X0, G


def oracle_run(wl, X0, G, steps, first=0):
    """Evolves (X, V) with the oracle for ``steps`` iterations; returns X, V
    (fp64) and the list of per-step masks."""
    n, m = wl.n, wl.m
    X = X0.astype(np.float64)
    V = np.zeros_like(X)
    mixer = OracleMixer(wl)
    d = oracle_delay(wl)
    lr, mu = float(np.float32(wl.lr)), float(np.float32(wl.momentum))
    masks = []
    for k in range(first, first + steps):
        s = oracle.schedule.sample_schedule(wl.seed, k, n, m, d)
        masks.append(s["mask"])
        X, V = oracle.step.step(X, V, G, s["mask"], mixer.w(k), lr, mu, ORACLE_ORDER[wl.order])
    return X, V, masks




def mlp_blocks(d_in, hidden, classes):
    """(name, start, stop) of the W1, b1, W2, b2 blocks of a flat MLP vector."""
    b1 = d_in * hidden
    w2 = b1 + hidden
    b2 = w2 + hidden * classes
    return [("W1", 0, b1), ("b1", b1, w2), ("W2", w2, b2), ("b2", b2, b2 + classes)]


def pad_cols(X, P):
    """X with zero columns appended up to P (the library pads the flat MLP
    vector to a multiple of 4 floats; the oracle's vector is unpadded)."""
    X = np.asarray(X)
    out = np.zeros(X.shape[:-1] + (P,), X.dtype)
    out[..., :X.shape[-1]] = X
    return out


def rel_err_blocks(got, want, blocks) -> float:
    """Largest per-block rel_err along the last axis: each parameter block is
    measured against its own rms, so blocks of very different scale (1.57M
    first-layer weights beside 10 output biases) do not hide or inflate each
    other."""
    got = np.asarray(got)
    want = np.asarray(want)
    return max(rel_err(got[..., a:b], want[..., a:b]) for _, a, b in blocks)
