"""End-to-end workload: a two-layer MLP trained by Non-blocking D-PSGD.

The objective is the mean softmax cross-entropy of a 3072 -> 512 (ReLU) -> 10
network (Eq. 1 with l the per-sample loss).  For each finished mini-batch the
learner computes the gradient of the mini-batch's mean loss at its own replica
(Alg. 2, gradient line of the mini-batch loop).  Local data
and sampling follow the initialisation line of Alg. 1/2: the data set is split
into n equal shards, learner i owns shard i, and the shard is reshuffled at
the start of every local epoch (Sec. 3.2, shuffling bullet).

Flat parameter layout (the replica rows X[i] of the step): W1[d_in][hidden]
row-major at 0, b1 at d_in*hidden, W2[hidden][classes] at d_in*hidden+hidden,
b2 at d_in*hidden + hidden + hidden*classes.

Precision modes:
* exact:   every product and sum in fp64.
* bf16:    every GEMM input is first rounded to bf16 (round to nearest even,
           from the value's fp32 rounding), then multiplied and summed in
           fp64; bias, ReLU, softmax and cross-entropy stay fp64.  The GEMMs
           are Z1 = A W1, Z2 = H W2, dW2 = H^T dZ2, dH = dZ2 W2^T and
           dW1 = A^T dZ1; the bias gradients are plain sums.

Pins (tests/test_oracle_mlp.py): finite differences and torch.autograd in
exact mode, the Sec. 5.1 identity (the mean of equal-size mini-batch gradients
is the joint-batch gradient), bf16 rounding against torch's bfloat16 cast, the
initial loss near ln(classes), and permutation invariants of the shuffle.
Pins of ``train`` (tests/test_oracle_mlp_train.py), each against torch
autograd in float64: with every mini-batch finished and uniform W it is
synchronous SGD with momentum on the joint batch of the learners' windows
(Sec. 5.1 with Eq. 2), evaluation losses included; with partial masks and no
momentum one iteration is SGD on the finished samples only; the first
mix-then-step iteration is each learner's own SGD step with lr c_i / m; the
workload's mixing kind is the one applied.
"""

from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from . import philox

EXACT = "exact"
BF16 = "bf16"


@dataclass(frozen=True)
class Shape:
    d_in: int = 3072
    hidden: int = 512
    classes: int = 10
    batch: int = 32

    @property
    def n_params(self) -> int:
        return self.d_in * self.hidden + self.hidden + self.hidden * self.classes + self.classes

    def offsets(self):
        w1 = 0
        b1 = self.d_in * self.hidden
        w2 = b1 + self.hidden
        b2 = w2 + self.hidden * self.classes
        return w1, b1, w2, b2


def bf16_round(x) -> np.ndarray:
    """Round to bfloat16 (nearest, ties to even) through the value's fp32
    rounding; returned as fp64 holding the bf16 value exactly."""
    f = np.ascontiguousarray(np.asarray(x, dtype=np.float32))
    u = f.view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = ((u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)) << np.uint64(16)
    return r.astype(np.uint32).view(np.float32).astype(np.float64)


def _g(x, mode):
    return bf16_round(x) if mode == BF16 else np.asarray(x, dtype=np.float64)


def unpack(params, s: Shape):
    p = np.asarray(params, dtype=np.float64)
    w1, b1, w2, b2 = s.offsets()
    return (p[w1:b1].reshape(s.d_in, s.hidden), p[b1:w2], p[w2:b2].reshape(s.hidden, s.classes),
            p[b2:b2 + s.classes])


def forward(params, A, y, s: Shape, mode: str = BF16):
    """Mean cross-entropy of the mini-batch (A[b][d_in], labels y[b]) and the
    intermediates the backward pass needs."""
    W1, b1, W2, b2 = unpack(params, s)
    Z1 = _g(A, mode) @ _g(W1, mode) + b1
    H = np.maximum(Z1, 0.0)
    Z2 = _g(H, mode) @ _g(W2, mode) + b2
    zmax = Z2.max(axis=1, keepdims=True)
    lse = zmax[:, 0] + np.log(np.exp(Z2 - zmax).sum(axis=1))
    rows = np.arange(len(y))
    loss = float(np.mean(lse - Z2[rows, y]))
    return loss, dict(Z1=Z1, H=H, Z2=Z2, lse=lse)


def grad(params, A, y, s: Shape, mode: str = BF16):
    """(flat gradient of the mini-batch mean loss, that loss)."""
    W1, b1, W2, b2 = unpack(params, s)
    loss, c = forward(params, A, y, s, mode)
    b = len(y)
    P = np.exp(c["Z2"] - c["lse"][:, None])
    onehot = np.zeros_like(P)
    onehot[np.arange(b), y] = 1.0
    dZ2 = (P - onehot) / b
    dW2 = _g(c["H"], mode).T @ _g(dZ2, mode)
    db2 = dZ2.sum(axis=0)
    dH = _g(dZ2, mode) @ _g(W2, mode).T
    dZ1 = dH * (c["Z1"] > 0.0)
    dW1 = _g(A, mode).T @ _g(dZ1, mode)
    db1 = dZ1.sum(axis=0)
    return np.concatenate([dW1.reshape(-1), db1, dW2.reshape(-1), db2]), loss


# --------------------------------------------------------------- local shuffle
class Shuffler:
    """Sample indices of learner i's mini-batches (Alg. 1/2 initialisation and
    shuffling step).  Learner i owns samples [shard*i, shard*(i+1)).  Local
    epoch e is a Fisher-Yates permutation of the shard (from the top: position
    t swaps with a uniform position in [0, t], drawn from Philox word 0 at
    counter (e, i, t) under key (seed, 4)); iteration k of the epoch takes the
    k-th consecutive window of m*b permuted samples and mini-batch j is the
    j-th run of b samples in that window.  A window is consumed whether or not
    its mini-batches finish (abandoned mini-batches are skipped, not
    re-queued); shard mod (m*b) left-over samples are dropped each epoch."""

    def __init__(self, seed: int, shard: int, m: int, b: int):
        self.seed, self.shard, self.m, self.b = seed, shard, m, b
        self.per_epoch = shard // (m * b)
        if self.per_epoch < 1:
            raise ValueError("shard smaller than one iteration's samples")
        self._cache = {}

    def permutation(self, epoch: int, learner: int) -> np.ndarray:
        hit = self._cache.get(learner)
        if hit is None or hit[0] != epoch:  # keep the current epoch of each learner
            perm = list(range(self.shard))
            for t in range(self.shard - 1, 0, -1):
                r = philox.bounded(philox.word(self.seed, philox.PURPOSE_SHUFFLE, epoch, learner, t),
                                   t + 1)
                perm[t], perm[r] = perm[r], perm[t]
            hit = (epoch, np.array(perm, dtype=np.int64))
            self._cache[learner] = hit
        return hit[1]

    def indices(self, step: int, learner: int) -> np.ndarray:
        """Global sample indices [m][b] of learner ``learner`` at iteration ``step``."""
        e, w = divmod(step, self.per_epoch)
        perm = self.permutation(e, learner)
        win = perm[w * self.m * self.b:(w + 1) * self.m * self.b]
        return (win + self.shard * learner).reshape(self.m, self.b)


# ------------------------------------------------------------------ training
def train(wl, A, y, x0, steps: int, mode: str = BF16, log=None, blocking: bool = False,
          evaluate: bool = True, stop=None):
    """Non-blocking decentralized SGD on the MLP (Alg. 2): every iteration
    draws the schedule, computes the gradient of each finished mini-batch at
    the learner's own replica, then mixes and steps with the workload's W
    (``wl.mixing``: uniform for ring all-reduce, ring for D-PSGD, matcha for
    MATCHA's random matchings) in the workload's order.

    ``wl`` carries n, m, batch, the shape, delay model, mixing kind, order,
    lr, momentum, seed and the evaluation cadence; A[samples][d_in] and y are
    the data, x0 the common initial replica (Alg. 1/2 initialisation).
    ``blocking``: the synchronous baseline on the same W and data, every
    mini-batch finished and each iteration charged the slowest learner's
    time.  Returns a dict with per-step mean losses (over learners, of the
    mean over their finished mini-batches), evaluation losses of the average
    replica (the method's output, Alg. 1/2) every ``wl.eval_every`` steps and
    at the end (when ``evaluate``), per-step finished counts and simulated
    seconds, and the final X and V (fp64).  ``stop`` (optional) is called
    after each iteration with its index and ends training early when it
    returns True.
    """
    from . import schedule, step as step_mod, workload

    s = Shape(wl.d_in, wl.hidden, wl.classes, wl.batch)
    n, m, P = wl.n, wl.m, s.n_params
    d = workload.delay(wl)
    mixer = workload.mixer(wl)
    order = workload.order(wl)
    lr, mu = float(np.float32(wl.lr)), float(np.float32(wl.momentum))
    shuf = Shuffler(wl.seed, wl.n_samples // n, m, wl.batch)
    X = np.tile(np.asarray(x0, dtype=np.float64), (n, 1))
    V = np.zeros_like(X)
    ev_idx = wl.eval_indices()
    out = dict(step_loss=[], counts=[], eval_step=[], eval_loss=[], seconds=[])

    def evaluate_mean(k):
        xbar = X.mean(axis=0)
        losses = [forward(xbar, A[ev_idx[r:r + s.batch]], y[ev_idx[r:r + s.batch]], s, mode)[0]
                  for r in range(0, len(ev_idx), s.batch)]
        out["eval_step"].append(k)
        out["eval_loss"].append(float(np.mean(losses)))

    G = np.zeros((n, m, P))
    k = 0
    for k in range(steps):
        if evaluate and k % wl.eval_every == 0:
            evaluate_mean(k)
        sch = schedule.sample_schedule(wl.seed, k, n, m, d)
        if blocking:
            sch["mask"] = np.ones((n, m), dtype=np.uint8)
            sch["counts"] = np.full(n, m, dtype=np.int32)
            out["seconds"].append(sch["t_sync"])
        else:
            out["seconds"].append(sch["t_step"])
        learner_losses = []
        for i in range(n):
            idx = shuf.indices(k, i)
            ls = []
            for j in range(m):
                if sch["mask"][i, j]:
                    G[i, j], loss = grad(X[i], A[idx[j]], y[idx[j]], s, mode)
                    ls.append(loss)
            learner_losses.append(np.mean(ls))
        out["step_loss"].append(float(np.mean(learner_losses)))
        out["counts"].append(sch["counts"].copy())
        X, V = step_mod.step(X, V, G, sch["mask"], mixer.w(k), lr, mu, order)
        if log:
            log(k, out["step_loss"][-1])
        if stop is not None and stop(k):
            k += 1
            break
    else:
        k = steps
    if evaluate:
        evaluate_mean(k)
    out["X"], out["V"] = X, V
    out["iterations"] = len(out["step_loss"])
    return out
