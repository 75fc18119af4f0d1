"""Pins for the oracle's MLP training loop (``oracle.mlp.train``): its
composition of shards and shuffle windows, finished-only gradients, the
count-normalised accumulation, the learning rate lr * c_i / m, the step and
the evaluation of the average replica, each checked against an independent
PyTorch (autograd, float64) computation fixed by the paper:

* Sec. 5.1 with Eq. 2: with every mini-batch finished and uniform W (ring
  all-reduce), stepping then averaging keeps the replicas equal, and the
  iteration is synchronous SGD with momentum on the joint batch of all
  learners' windows (``torch.optim.SGD``).  With n = 3 the D-PSGD ring is the
  same W.
* With partial masks, no momentum and uniform W, one iteration is plain SGD
  on the mean cross-entropy of the finished samples only, scaled by
  1 / (n m b): a learner's step lr (c_i / m) (1 / c_i) sum of finished
  gradients adds up to lr / m times its finished sum.
* MIX_THEN_STEP from identical replicas: the first iteration leaves learner i
  at x0 - lr (c_i / m) g_i, per-learner SGD on its own finished samples.
* The mixing kind of the workload is honoured: MATCHA's W (oracle.mixing) and
  the ring give different replicas after the second iteration.
"""

import dataclasses

import numpy as np
import pytest
import torch

from oracle import mlp, schedule
from oracle.mlp import EXACT, Shape
from synth import mlp_data, workloads


def _wl(**kw):
    base = dict(n=3, m=2, batch=32, d_in=16, hidden=8, classes=3, n_samples=3 * 160,
                mixing="uniform", order=workloads.STEP_THEN_MIX,
                delay=workloads.DelaySpec("const", 1.0, 0.0), lr=0.1, momentum=0.9, steps=5,
                eval_every=2, eval_samples=64, eval_stride=7)
    base.update(kw)
    return workloads.MlpWorkload("pin", **base)


def _data(wl):
    A = mlp_data.inputs(3, wl.n_samples, wl.d_in)
    y = mlp_data.teacher_labels(3, A, wl.hidden, wl.classes)
    x0 = mlp_data.student_init(3, wl.d_in, wl.hidden, wl.classes)
    return A, y, x0


def _model(params, s):
    p = torch.tensor(np.asarray(params, dtype=np.float64), dtype=torch.float64, requires_grad=True)
    return p


def _ce(p, A, y, s, reduction="mean"):
    w1, b1, w2, b2 = s.offsets()
    W1 = p[w1:b1].view(s.d_in, s.hidden)
    W2 = p[w2:b2].view(s.hidden, s.classes)
    H = torch.relu(torch.as_tensor(np.asarray(A, dtype=np.float64)) @ W1 + p[b1:w2])
    logits = H @ W2 + p[b2:b2 + s.classes]
    return torch.nn.functional.cross_entropy(logits, torch.as_tensor(np.asarray(y), dtype=torch.long),
                                             reduction=reduction)


# The ABI stores W in fp32, and the oracle mixes with the fp32 entries widened
# to fp64 (as the library does): 1/4 is exact, fp32(1/3) is 1/3 + 1e-8, whose
# rows sum to 1 + 3e-8, so the n = 3 ring case carries that scale per step.
@pytest.mark.parametrize("mixing,n,rtol", [("uniform", 4, 1e-11), ("ring", 3, 1e-6)])
def test_full_mask_allreduce_is_synchronous_sgd_with_momentum(mixing, n, rtol):
    wl = _wl(mixing=mixing, n=n, n_samples=n * 160)  # n = 3: the ring is J/3
    s = Shape(wl.d_in, wl.hidden, wl.classes, wl.batch)
    A, y, x0 = _data(wl)
    out = mlp.train(wl, A, y, x0, wl.steps, mode=EXACT)
    assert all((c == wl.m).all() for c in out["counts"])

    p = _model(x0, s)
    opt = torch.optim.SGD([p], lr=float(np.float32(wl.lr)), momentum=float(np.float32(wl.momentum)))
    shuf = mlp.Shuffler(wl.seed, wl.n_samples // wl.n, wl.m, wl.batch)
    ev = wl.eval_indices()
    ev_loss = []
    for k in range(wl.steps):
        if k % wl.eval_every == 0:
            ev_loss.append(float(_ce(p, A[ev], y[ev], s).detach()))
        joint = np.concatenate([shuf.indices(k, i).reshape(-1) for i in range(wl.n)])
        opt.zero_grad()
        loss = _ce(p, A[joint], y[joint], s)
        loss.backward()
        opt.step()
        assert out["step_loss"][k] == pytest.approx(float(loss.detach()), rel=rtol), k
    ev_loss.append(float(_ce(p, A[ev], y[ev], s).detach()))
    want = p.detach().numpy()
    for i in range(wl.n):  # every replica equals the synchronous model
        np.testing.assert_allclose(out["X"][i], want, rtol=rtol, atol=1e-13)
    np.testing.assert_allclose(out["eval_loss"], ev_loss, rtol=rtol)
    assert out["eval_step"] == [0, 2, 4, 5]


def test_partial_masks_step_on_finished_samples_only():
    wl = _wl(n=4, m=4, n_samples=4 * 256, momentum=0.0, steps=1,
             delay=workloads.DelaySpec("exp", 1.0, 1.0))
    s = Shape(wl.d_in, wl.hidden, wl.classes, wl.batch)
    A, y, x0 = _data(wl)
    sch = schedule.sample_schedule(wl.seed, 0, wl.n, wl.m, schedule.Delay(schedule.DELAY_EXP, 1.0, 1.0))
    assert 0 < sch["mask"].sum() < wl.n * wl.m  # a partial mask
    out = mlp.train(wl, A, y, x0, 1, mode=EXACT, evaluate=False)
    assert np.array_equal(out["counts"][0], sch["counts"])

    shuf = mlp.Shuffler(wl.seed, wl.n_samples // wl.n, wl.m, wl.batch)
    rows = np.concatenate([shuf.indices(0, i)[j] for i in range(wl.n) for j in range(wl.m)
                           if sch["mask"][i, j]])
    p = _model(x0, s)
    opt = torch.optim.SGD([p], lr=float(np.float32(wl.lr)))
    (_ce(p, A[rows], y[rows], s, "sum") / (wl.n * wl.m * wl.batch)).backward()
    opt.step()
    for i in range(wl.n):
        np.testing.assert_allclose(out["X"][i], p.detach().numpy(), rtol=1e-11, atol=1e-13)


@pytest.mark.parametrize("mixing,n,rtol", [("uniform", 4, 1e-11), ("ring", 5, 1e-6)])
def test_mix_then_step_first_iteration_is_per_learner_sgd(mixing, n, rtol):
    wl = _wl(n=n, m=4, n_samples=n * 256, mixing=mixing, order=workloads.MIX_THEN_STEP, steps=1,
             delay=workloads.DelaySpec("exp", 1.0, 1.0))
    s = Shape(wl.d_in, wl.hidden, wl.classes, wl.batch)
    A, y, x0 = _data(wl)
    out = mlp.train(wl, A, y, x0, 1, mode=EXACT, evaluate=False)
    counts = out["counts"][0]
    assert len(set(counts.tolist())) > 1  # learners finished different numbers
    shuf = mlp.Shuffler(wl.seed, wl.n_samples // wl.n, wl.m, wl.batch)
    for i in range(wl.n):
        rows = shuf.indices(0, i)[:counts[i]].reshape(-1)  # the finished prefix
        p = _model(x0, s)
        # lr (c/m) times the mean over the finished mini-batches = lr/(m b) times the sum
        opt = torch.optim.SGD([p], lr=float(np.float32(wl.lr)) / (wl.m * wl.batch))
        _ce(p, A[rows], y[rows], s, "sum").backward()
        opt.step()
        np.testing.assert_allclose(out["X"][i], p.detach().numpy(), rtol=rtol, atol=1e-13)
        # momentum buffer after one step: the learner's mean finished gradient
        np.testing.assert_allclose(out["V"][i], p.grad.numpy() / (counts[i] * wl.batch),
                                   rtol=1e-10, atol=1e-14)


def test_mixing_kind_is_honoured():
    wl = _wl(n=8, m=2, n_samples=8 * 128, order=workloads.MIX_THEN_STEP, steps=2,
             delay=workloads.DelaySpec("exp", 1.0, 1.0))
    A, y, x0 = _data(wl)
    runs = {k: mlp.train(dataclasses.replace(wl, mixing=k), A, y, x0, 2, mode=EXACT, evaluate=False)
            for k in ("ring", "matcha", "uniform")}
    # the same first iteration (identical replicas mix to themselves) ...
    one = {k: mlp.train(dataclasses.replace(wl, mixing=k), A, y, x0, 1, mode=EXACT, evaluate=False)
           for k in ("ring", "matcha", "uniform")}
    # (up to the ring's fp32(1/3) weights, whose rows sum to 1 + 3e-8)
    np.testing.assert_allclose(one["ring"]["X"], one["matcha"]["X"], rtol=1e-6, atol=1e-7)
    np.testing.assert_allclose(one["uniform"]["X"], one["matcha"]["X"], rtol=1e-12, atol=1e-15)
    # ... then different W give different replicas
    assert np.abs(runs["ring"]["X"] - runs["matcha"]["X"]).max() > 1e-6
    assert np.abs(runs["ring"]["X"] - runs["uniform"]["X"]).max() > 1e-6
    # uniform W (J/8, exact in fp32), mix-then-step: after the second iteration
    # every learner sits at the mean of the first iteration's replicas minus
    # its own step eta_i v_i
    lr = float(np.float32(wl.lr))
    u = runs["uniform"]
    want = one["uniform"]["X"].mean(axis=0)[None, :] - np.array(
        [lr * c / wl.m * v for c, v in zip(u["counts"][1], u["V"])])
    np.testing.assert_allclose(u["X"], want, rtol=1e-12, atol=1e-15)
