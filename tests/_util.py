"""Shared test helpers: the parity metric and oracle-side drivers."""

from __future__ import annotations

import numpy as np

import oracle
import oracle.workload

# Parity bar for fp32 results: max_k |got_k - want_k| / max(|want_k|, rms(want))
# over each tensor (X and V separately).  Stated for the step in fp32 against
# the fp64 oracle; the max(|want|, rms) floor keeps near-zero elements from
# turning rounding noise into huge relative errors.
TOL = 1e-5

ORACLE_ORDER = oracle.workload.ORDERS
oracle_delay = oracle.workload.delay
window_inputs = oracle.workload.window_inputs


def rel_err(got, want) -> float:
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    if want.size == 0:
        return 0.0
    rms = float(np.sqrt(np.mean(want * want)))
    denom = np.maximum(np.abs(want), rms if rms > 0 else 1.0)
    return float(np.max(np.abs(got - want) / denom))


def OracleMixer(wl):
    """The oracle's per-iteration W of a workload (fp32-rounded, widened)."""
    return oracle.workload.mixer(wl)


def oracle_run(wl, X0, G, steps, first=0):
    """Evolves (X, V) with the oracle for ``steps`` iterations; returns X, V
    (fp64) and the list of per-step masks."""
    return oracle.workload.run(wl, X0, G, steps, first)


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
