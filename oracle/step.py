"""One Non-blocking iteration on n learner replicas (Alg. 2, averaging and
update steps; Sec. 3.2, the learning-rate, gradient, averaging and update
bullets), plus heavy-ball momentum.

Shapes: X[n, P] replicas, V[n, P] momentum buffers, G[n, m, P] per-mini-batch
gradients, mask[n, m] (nonzero = finished before the terminal signal),
W[n, n] mixing matrix.  All arithmetic is fp64; fp32 inputs are widened first.

Readings (the paper is silent or inconsistent on these):

* accumulated gradient = mean over the finished mini-batches; learning rate
  lr * c_i / m with c_i the finished count (Sec. 3.2 learning-rate bullet).
  Without momentum the step is therefore (lr / m) * (sum of finished
  mini-batch gradients), and with every mini-batch finished it is lr times the
  large-batch gradient (Sec. 5.1).
* momentum (not in the paper): v_i <- mu * v_i + g_i, then the learner's
  learning rate multiplies v_i; v is local and never mixed; no dampening.
* order: MIX_THEN_STEP mixes the pre-step models and subtracts the local step
  (Alg. 2 as printed); STEP_THEN_MIX steps first and mixes the stepped models
  (Eq. 4-6 and Alg. 3).
"""

from __future__ import annotations

import numpy as np

MIX_THEN_STEP = 0
STEP_THEN_MIX = 1


def finished_counts(mask) -> np.ndarray:
    mask = np.asarray(mask)
    n, m = mask.shape
    counts = np.zeros(n, dtype=np.int64)
    for i in range(n):
        for j in range(m):
            if mask[i, j]:
                counts[i] += 1
    return counts


def accumulate(G, mask) -> np.ndarray:
    """g_i = (1 / c_i) * sum of G[i, j] over the finished mini-batches j."""
    G = np.asarray(G)
    n, m, P = G.shape
    out = np.zeros((n, P), dtype=np.float64)
    for i in range(n):
        acc = np.zeros(P, dtype=np.float64)
        c = 0
        for j in range(m):
            if mask[i][j]:
                acc = acc + G[i, j].astype(np.float64)
                c += 1
        if c == 0:
            raise ValueError(f"learner {i} finished no mini-batch")
        out[i] = acc / c
    return out


def learning_rates(counts, m: int, lr: float) -> np.ndarray:
    """eta_i = lr * c_i / m: a learner that finished more mini-batches takes a
    larger step (Sec. 3.2, learning-rate bullet)."""
    return np.array([float(lr) * float(c) / float(m) for c in counts], dtype=np.float64)


def momentum(V, g, mu: float) -> np.ndarray:
    return float(mu) * np.asarray(V, dtype=np.float64) + g


def mix(W, Z) -> np.ndarray:
    """z'_i = sum_p W[i, p] z_p (Alg. 2 averaging step)."""
    return np.asarray(W, dtype=np.float64) @ np.asarray(Z, dtype=np.float64)


def step(X, V, G, mask, W, lr: float, mu: float, order: int):
    """Returns (X', V') in fp64."""
    G = np.asarray(G)
    n, m, _ = G.shape
    counts = finished_counts(mask)
    g = accumulate(G, mask)
    eta = learning_rates(counts, m, lr)
    V_new = momentum(V, g, mu)
    X = np.asarray(X, dtype=np.float64)
    if order == MIX_THEN_STEP:
        X_new = mix(W, X) - eta[:, None] * V_new
    elif order == STEP_THEN_MIX:
        X_new = mix(W, X - eta[:, None] * V_new)
    else:
        raise ValueError(f"unknown order {order}")
    return X_new, V_new


def parameter_server_step(x_ps, V, G, mask, lr: float, mu: float):
    """Non-blocking synchronous centralized SGD (Alg. 3): every learner
    computes its accumulated gradient at the server's model, the server
    subtracts the learners' lr * c_i / m scaled steps, averaged over the n
    learners (Alg. 3 omits the 1/n of Eq. 2; it is restored here), and every
    learner takes the new server model.  With momentum, each learner keeps its
    own buffer v_i <- mu v_i + g_i and contributes eta_i v_i.

    x_ps: [P]; V: [n, P]; G: [n, m, P].  Returns (x_ps', V') in fp64."""
    G = np.asarray(G)
    n, m, _ = G.shape
    counts = finished_counts(mask)
    g = accumulate(G, mask)
    eta = learning_rates(counts, m, lr)
    V_new = momentum(V, g, mu)
    x = np.asarray(x_ps, dtype=np.float64).copy()
    for i in range(n):
        x = x - (eta[i] / n) * V_new[i]
    return x, V_new
