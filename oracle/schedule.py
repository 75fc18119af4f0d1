"""Simulated straggler schedule: per-mini-batch times, the terminal signal and
the finished-mini-batch mask of one iteration (Alg. 2, the mini-batch loop;
Lemma 1 and Thm 2 for the timing model).

Each learner processes its N mini-batches in order.  The first learner to
finish all of them broadcasts the terminal signal (Alg. 2, the branch taken
when a learner's count reaches N); every learner keeps the mini-batches it
finished by then and abandons the rest.  With the times of learner i written t[i, 0..m-1] and their
running sums C[i, j], the signal time is T = min_i C[i, m-1] and learner i keeps
mini-batches j with C[i, j] <= T (finished by the signal time, boundary
included).  A learner that finished none keeps its first one (the step is
undefined for zero finished mini-batches), which extends the iteration to that
learner's first finish time.

Delay models (rate convention for Exp, mean 1/rate, as in Remark 1 of App. A):

* CONST:  D = 0
* EXP:    D = -log(u) / rate
* LOMAX:  D = u**(-1/shape) - 1   (so base 1 plus D is Pareto with scale 1)

t[i, j] = s_i * (base + D) where s_i is ``slow_factor`` for the one slowed
learner and 1 otherwise, or, with ``slow_learner = SLOW_RANDOM``, the paper's
heterogeneity model (Sec. 6.1: which nodes are slowed and by how much changes
every iteration, the slowest taking up to twice as long): every iteration
each learner is slowed with probability ``slow_prob`` by a factor uniform
between 1 and ``slow_factor`` (Philox words 0 and 1 at counter (step, i, 0, 0)
under key (seed, 5)).

The delay variate u of mini-batch j comes from Philox word 0 at counter
(step, i, j, 0) under key (seed, 1).  Scalar ``math.log`` / ``math.pow`` are
used on purpose (the platform libm, one value at a time).
"""

from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

from . import philox

DELAY_CONST = 0
DELAY_EXP = 1
DELAY_LOMAX = 2
SLOW_NONE = -1
SLOW_RANDOM = -2


@dataclass(frozen=True)
class Delay:
    kind: int = DELAY_EXP
    base: float = 1.0
    param: float = 1.0          # EXP: rate; LOMAX: shape
    slow_learner: int = -1      # -1: nobody is slowed; -2: random per iteration
    slow_factor: float = 1.0
    slow_prob: float = 0.0      # random slow-down only


def minibatch_time(seed: int, step: int, i: int, j: int, d: Delay) -> float:
    """Wall time of learner i on mini-batch j of iteration ``step``."""
    u = philox.u01(philox.word(seed, philox.PURPOSE_DELAY, step, i, j))
    if d.kind == DELAY_CONST:
        extra = 0.0
    elif d.kind == DELAY_EXP:
        extra = -math.log(u) / d.param
    elif d.kind == DELAY_LOMAX:
        extra = math.pow(u, -1.0 / d.param) - 1.0
    else:
        raise ValueError(f"unknown delay kind {d.kind}")
    return slowdown(seed, step, i, d) * (d.base + extra)


def slowdown(seed: int, step: int, i: int, d: Delay) -> float:
    """s_i of learner i in iteration ``step``."""
    if d.slow_learner == SLOW_RANDOM:
        w0, w1, _, _ = philox.block((step, i, 0, 0), (seed, philox.PURPOSE_SLOWDOWN))
        if philox.u01(w0) < d.slow_prob:
            return 1.0 + (d.slow_factor - 1.0) * philox.u01(w1)
        return 1.0
    return d.slow_factor if i == d.slow_learner else 1.0


def sample_schedule(seed: int, step: int, n: int, m: int, d: Delay) -> dict:
    """One iteration's schedule.

    Returns a dict with ``times`` f64[n, m], ``finish`` f64[n, m] (running
    sums), ``deadline`` T, ``counts`` int32[n], ``mask`` uint8[n, m] (1 =
    finished), ``t_sync`` (time the slowest learner would need for all m, the
    blocking baseline's iteration time) and ``t_step`` (this iteration's time
    including any forced first mini-batch).
    """
    times = np.zeros((n, m), dtype=np.float64)
    finish = np.zeros((n, m), dtype=np.float64)
    for i in range(n):
        running = 0.0
        for j in range(m):
            t = minibatch_time(seed, step, i, j, d)
            running = running + t
            times[i, j] = t
            finish[i, j] = running
    deadline = min(finish[i, m - 1] for i in range(n))
    counts = np.zeros(n, dtype=np.int32)
    mask = np.zeros((n, m), dtype=np.uint8)
    for i in range(n):
        done = 0
        for j in range(m):
            if finish[i, j] <= deadline:
                done += 1
        c = max(1, done)
        counts[i] = c
        for j in range(c):
            mask[i, j] = 1
    t_sync = max(finish[i, m - 1] for i in range(n))
    t_step = max(deadline, max(finish[i, counts[i] - 1] for i in range(n)))
    return dict(times=times, finish=finish, deadline=deadline, counts=counts, mask=mask,
                t_sync=t_sync, t_step=t_step)


def accounting(times) -> dict:
    """Sec. 4.3 accounting of one iteration from its per-mini-batch times
    t[n, m] (the schedule's ``times``), in units of mini-batches (the batch
    B is the m mini-batches of a learner).

    Learner i's time for its whole batch is X_i = sum_j t[i, j] (summed in
    mini-batch order, as the schedule's running sums); X_{k:P} is the k-th
    smallest of the X_i, and Y = sum_k 1 / X_{k:P}, summed from the fastest
    to the slowest learner.  Then:

    * ``throughput``       Thm 3: B * Y, each learner's B / X_i added up;
    * ``throughput_sync``  Thm 4: P * B / X_{P:P}, the blocking baseline's;
    * ``data``             Cor. 1: B * Y * X_{1:P}, the (fractional) amount
                           of data trained in one non-blocking iteration,
                           which lasts X_{1:P}, when every learner runs at a
                           constant speed within the iteration;
    * ``ratio``            Thm 5: Y * X_{P:P} / P, the non-blocking over
                           the blocking throughput.

    Pins (tests/test_oracle_schedule.py): equal times give Y X_{1:P} = P and a
    ratio of 1; under constant per-learner speeds (DELAY_CONST with the
    random slow-down) the schedule's finished counts lie within P of the
    Cor. 1 amount, below it; the ratio is at least 1 and equals Thm 3 over
    Thm 4.
    """
    times = np.asarray(times, dtype=np.float64)
    n, m = times.shape
    X = []
    for i in range(n):
        total = 0.0
        for j in range(m):
            total = total + float(times[i, j])
        if not total > 0.0:
            raise ValueError(f"learner {i} has a non-positive batch time")
        X.append(total)
    order_stats = sorted(X)
    Y = 0.0
    for x in order_stats:
        Y = Y + 1.0 / x
    x_first, x_last = order_stats[0], order_stats[-1]
    throughput = m * Y
    return dict(x_first=x_first, x_last=x_last, y=Y, throughput=throughput,
                throughput_sync=(n * m) / x_last, data=throughput * x_first,
                ratio=(Y * x_last) / n)
