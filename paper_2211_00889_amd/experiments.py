"""Simulated time-to-loss: Non-blocking decentralized SGD (Alg. 2) against its
synchronous baseline on the end-to-end MLP workload, for each of the paper's
three mixing kinds (Sec. 6.2): D-PSGD on the ring (Eq. 6), MATCHA's random
matchings, and ring all-reduce (uniform W, Eq. 4-5).  Same kernels, same data
and shuffles, same W sequence for both runs of a kind.

Each iteration is charged its simulated wall time: the non-blocking step
waits for the terminal signal (T_step), the baseline for the slowest learner
to finish all m mini-batches (T_sync).  The loss of the average replica is
evaluated every ``eval_every`` iterations.  The per-iteration time ratio is
the one-GPU analogue of Thm 1 (E[X_{1:P}] / E[X_{P:P}]); the time to reach a
loss level is the analogue of the paper's comparison of time to a given
training loss (Sec. 6.2), here on synthetic data.  Every non-blocking
iteration also logs the Sec. 4.3 accounting of its schedule
(``nbsgd_iteration_accounting``): the finished mini-batches beside Cor. 1's
constant-speed amount B Y X_{1:P}, and the Thm 5 throughput ratio
Y X_{P:P} / P.

    python -m paper_2211_00889_amd.experiments --workload hetero --mixing all --steps 200
"""

from __future__ import annotations

import argparse
import json

import numpy as np


def run(wl, steps: int, blocking: bool, device="cuda:0", data=None, labels=None, x0=None):
    import torch

    from . import _lib
    from .runner import MlpRunner

    r = MlpRunner(wl, device, data, labels, x0)
    t, times, losses, samples, finished = 0.0, [], [], 0, []
    cor1, thm5 = [], []
    for k in range(steps + 1):
        if k % wl.eval_every == 0 or k == steps:
            times.append(t)
            losses.append(float(r.evaluate().mean().cpu()))
        if k == steps:
            break
        _, counts, seconds = r.step(k, blocking=blocking)
        t += seconds
        samples += int(counts.sum()) * wl.batch
        finished.append(int(counts.sum()))
        acc = _lib.iteration_accounting(r.last_schedule[2])
        cor1.append(acc["data"])
        thm5.append(acc["ratio"])
    torch.cuda.synchronize()
    return dict(time=times, eval_loss=losses, samples=samples, mean_finished=float(np.mean(finished)),
                mean_cor1_data=float(np.mean(cor1)), mean_thm5_ratio=float(np.mean(thm5)),
                seconds_per_iteration=t / steps)


def time_to(times, losses, level):
    """First simulated time at which the evaluation loss reaches ``level``,
    interpolating linearly between evaluations; None if never."""
    for k in range(len(losses)):
        if losses[k] <= level:
            if k == 0:
                return times[0]
            t0, t1, l0, l1 = times[k - 1], times[k], losses[k - 1], losses[k]
            return t0 + (t1 - t0) * (l0 - level) / (l0 - l1)
    return None


LEVELS = (1.5, 1.0, 0.7, 0.5)


def compare(wl, steps: int, data, labels, x0, levels=LEVELS) -> dict:
    """Non-blocking and synchronous runs of one workload; their time-to-loss."""
    nb = run(wl, steps, False, data=data, labels=labels, x0=x0)
    bl = run(wl, steps, True, data=data, labels=labels, x0=x0)
    out = {"workload": wl.name, "mixing": wl.mixing, "order": wl.order, "steps": steps,
           "nonblocking": nb, "blocking": bl,
           "time_per_iteration_ratio": bl["seconds_per_iteration"] / nb["seconds_per_iteration"],
           "time_to_loss": {}}
    for L in levels:
        a, b = time_to(nb["time"], nb["eval_loss"], L), time_to(bl["time"], bl["eval_loss"], L)
        out["time_to_loss"][str(L)] = {"nonblocking": a, "blocking": b,
                                       "speedup": (b / a) if (a and b) else None}
    return out


def main():
    from synth import mlp_data, workloads

    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", default="hetero", choices=["hetero", "exp"])
    ap.add_argument("--mixing", default="all", choices=["ring", "matcha", "uniform", "all"])
    ap.add_argument("--steps", type=int, default=200)
    args = ap.parse_args()
    base = workloads.MLP_HETERO if args.workload == "hetero" else workloads.MLP
    data = mlp_data.inputs(base.seed, base.n_samples, base.d_in)
    labels = mlp_data.teacher_labels(base.seed, data, base.hidden, base.classes)
    x0 = mlp_data.student_init(base.seed, base.d_in, base.hidden, base.classes)
    kinds = ["ring", "matcha", "uniform"] if args.mixing == "all" else [args.mixing]
    for kind in kinds:
        wl = workloads.mlp_with_mixing(base, kind)
        print(json.dumps(compare(wl, args.steps, data, labels, x0)), flush=True)


if __name__ == "__main__":
    main()
