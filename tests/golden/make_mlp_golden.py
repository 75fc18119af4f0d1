"""Writes tests/golden/mlp_trajectory.npz: the oracle's 200-step run of the
end-to-end MLP workload (bf16 GEMM inputs, fp64 arithmetic).  Calls only the
oracle and the input generator.  ``python tests/golden/make_mlp_golden.py``
(a few minutes on 8 cores)."""

import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

from oracle import mlp  # noqa: E402
from synth import mlp_data, workloads  # noqa: E402

OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "mlp_trajectory.npz")
N_SAMPLED = 4096  # final X / V compared at this many seeded positions per learner


def main():
    wl = workloads.MLP
    t0 = time.time()
    A = mlp_data.inputs(wl.seed, wl.n_samples, wl.d_in)
    y = mlp_data.teacher_labels(wl.seed, A, wl.hidden, wl.classes)
    x0 = mlp_data.student_init(wl.seed, wl.d_in, wl.hidden, wl.classes)
    print(f"inputs ready in {time.time() - t0:.1f} s", flush=True)
    res = mlp.train(wl, A, y, x0, wl.steps,
                    log=lambda k, l: print(f"step {k} loss {l:.5f} ({time.time() - t0:.0f} s)", flush=True)
                    if k % 10 == 0 else None)
    pos = np.sort(np.random.default_rng(1234).choice(wl.P, size=N_SAMPLED, replace=False))
    np.savez(OUT, step_loss=np.array(res["step_loss"]), counts=np.array(res["counts"], dtype=np.int32),
             eval_step=np.array(res["eval_step"]), eval_loss=np.array(res["eval_loss"]),
             positions=pos, X=res["X"][:, pos], V=res["V"][:, pos],
             label_counts=np.bincount(y, minlength=wl.classes).astype(np.int64),
             x0_sum=np.float64(np.sum(x0, dtype=np.float64)))
    print(f"wrote {OUT} in {time.time() - t0:.0f} s; final step loss {res['step_loss'][-1]:.5f}, "
          f"eval {res['eval_loss']}")


if __name__ == "__main__":
    main()
