"""Simulated time-to-loss: Non-blocking D-PSGD (Alg. 2) against its blocking
D-PSGD baseline (Eq. 6) on the end-to-end MLP workload, same kernels, same
ring W, same data and shuffles.

Each iteration is charged its simulated wall time: the non-blocking step
waits for the terminal signal (T_step), the baseline for the slowest learner
to finish all m mini-batches (T_sync).  The loss of the average replica is
evaluated every ``eval_every`` iterations.  The per-iteration time ratio is
the one-GPU analogue of Thm 1 (E[X_{1:P}] / E[X_{P:P}]); the time to reach a
loss level is the analogue of the paper's "up to 2x less time to the same
training loss" (Sec. 6.2), here on synthetic data.

    python -m paper_2211_00889_amd.experiments --workload hetero --steps 200
"""

from __future__ import annotations

import argparse
import json

import numpy as np


def run(wl, steps: int, blocking: bool, device="cuda:0", data=None, labels=None, x0=None):
    import torch

    from .runner import MlpRunner

    r = MlpRunner(wl, device, data, labels, x0)
    t, times, losses, samples, finished = 0.0, [], [], 0, []
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
    torch.cuda.synchronize()
    return dict(time=times, eval_loss=losses, samples=samples, mean_finished=float(np.mean(finished)),
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


def main():
    from synth import mlp_data, workloads

    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", default="hetero", choices=["hetero", "exp"])
    ap.add_argument("--steps", type=int, default=200)
    args = ap.parse_args()
    wl = workloads.MLP_HETERO if args.workload == "hetero" else workloads.MLP
    data = mlp_data.inputs(wl.seed, wl.n_samples, wl.d_in)
    labels = mlp_data.teacher_labels(wl.seed, data, wl.hidden, wl.classes)
    x0 = mlp_data.student_init(wl.seed, wl.d_in, wl.hidden, wl.classes)
    nb = run(wl, args.steps, False, data=data, labels=labels, x0=x0)
    bl = run(wl, args.steps, True, data=data, labels=labels, x0=x0)
    levels = [1.5, 1.0, 0.7, 0.5]
    out = {"workload": wl.name, "steps": args.steps,
           "nonblocking": nb, "blocking": bl,
           "time_per_iteration_ratio": bl["seconds_per_iteration"] / nb["seconds_per_iteration"],
           "time_to_loss": {}}
    for L in levels:
        a, b = time_to(nb["time"], nb["eval_loss"], L), time_to(bl["time"], bl["eval_loss"], L)
        out["time_to_loss"][str(L)] = {"nonblocking": a, "blocking": b,
                                       "speedup": (b / a) if (a and b) else None}
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
