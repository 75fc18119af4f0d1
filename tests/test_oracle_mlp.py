"""Pins for the MLP oracle: autograd and finite differences (exact mode), the
Sec. 5.1 identity, bf16 rounding against torch, initial loss, shuffle."""

import math

import numpy as np
import pytest
import torch

from oracle import mlp
from oracle.mlp import BF16, EXACT, Shape


def _problem(s: Shape, b: int, seed: int = 0):
    rng = np.random.default_rng(seed)
    params = rng.uniform(-0.5, 0.5, size=s.n_params)
    A = rng.standard_normal((b, s.d_in))
    y = rng.integers(0, s.classes, size=b)
    return params, A, y


def _torch_loss(params, A, y, s):
    p = torch.tensor(params, dtype=torch.float64, requires_grad=True)
    w1, b1, w2, b2 = s.offsets()
    W1 = p[w1:b1].view(s.d_in, s.hidden)
    W2 = p[w2:b2].view(s.hidden, s.classes)
    Ht = torch.relu(torch.tensor(A, dtype=torch.float64) @ W1 + p[b1:w2])
    logits = Ht @ W2 + p[b2:b2 + s.classes]
    loss = torch.nn.functional.cross_entropy(logits, torch.tensor(y, dtype=torch.long))
    loss.backward()
    return float(loss), p.grad.numpy()


def test_exact_gradient_matches_torch_autograd():
    s = Shape(d_in=24, hidden=16, classes=5, batch=8)
    params, A, y = _problem(s, 8)
    g, loss = mlp.grad(params, A, y, s, EXACT)
    tl, tg = _torch_loss(params, A, y, s)
    assert loss == pytest.approx(tl, rel=1e-12)
    np.testing.assert_allclose(g, tg, rtol=1e-10, atol=1e-13)


def test_exact_gradient_finite_differences():
    s = Shape(d_in=8, hidden=4, classes=3, batch=5)
    params, A, y = _problem(s, 5, seed=1)
    g, _ = mlp.grad(params, A, y, s, EXACT)
    h = 1e-6
    for k in range(s.n_params):
        e = np.zeros(s.n_params)
        e[k] = h
        fd = (mlp.forward(params + e, A, y, s, EXACT)[0] - mlp.forward(params - e, A, y, s, EXACT)[0]) / (2 * h)
        assert g[k] == pytest.approx(fd, rel=1e-5, abs=1e-8), k


def test_accumulated_minibatch_gradients_equal_joint_batch_gradient():
    # Sec. 5.1: with equal mini-batch sizes, the mean of the mini-batch mean-loss
    # gradients is the gradient of the joint batch's mean loss.
    s = Shape(d_in=12, hidden=8, classes=4, batch=6)
    params, A, y = _problem(s, 24, seed=2)
    parts = [mlp.grad(params, A[6 * j:6 * j + 6], y[6 * j:6 * j + 6], s, EXACT)[0] for j in range(4)]
    joint, _ = mlp.grad(params, A, y, s, EXACT)
    np.testing.assert_allclose(np.mean(parts, axis=0), joint, rtol=1e-11, atol=1e-14)


def test_bf16_round_matches_torch():
    rng = np.random.default_rng(3)
    x = np.concatenate([rng.standard_normal(100000).astype(np.float32) * 10.0 ** rng.integers(-30, 30, 100000),
                        np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -(1.0 + 2 ** -8), 0.0, -0.0,
                                  1.00390625, 1.01171875], dtype=np.float32)]).astype(np.float32)
    ours = mlp.bf16_round(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(ours, ref)


def test_bf16_mode_close_to_exact():
    s = Shape(d_in=64, hidden=32, classes=10, batch=32)
    params, A, y = _problem(s, 32, seed=4)
    params *= 0.2
    gb, lb = mlp.grad(params, A, y, s, BF16)
    ge, le = mlp.grad(params, A, y, s, EXACT)
    # bf16 keeps 8 significant bits: the loss moves by far less than 1%, the
    # gradient by a few percent rms (inputs rounded by up to 2^-9 each)
    assert abs(lb - le) < 1e-2 * abs(le)
    assert np.sqrt(np.mean((gb - ge) ** 2)) < 5e-2 * np.sqrt(np.mean(ge ** 2))
    assert not np.array_equal(gb, ge)


def test_initial_loss_near_log_classes():
    from synth import mlp_data

    s = Shape(d_in=3072, hidden=512, classes=10, batch=32)
    x0 = mlp_data.student_init(0)
    A = mlp_data.inputs(0, n_samples=64)
    y = np.arange(64) % 10
    loss, _ = mlp.forward(x0, A[:32], y[:32], s, BF16)
    assert abs(loss - math.log(10)) < 0.3


def test_shuffle_permutations_and_windows():
    sh = mlp.Shuffler(seed=5, shard=640, m=4, b=32)
    assert sh.per_epoch == 5
    for learner in (0, 3):
        seen = []
        for k in range(5):
            idx = sh.indices(k, learner)
            assert idx.shape == (4, 32)
            assert idx.min() >= 640 * learner and idx.max() < 640 * (learner + 1)
            seen.append(idx.reshape(-1))
        flat = np.concatenate(seen)
        assert len(set(flat.tolist())) == 640  # one epoch: every sample exactly once
        nxt = sh.indices(5, learner)            # next epoch: a new permutation
        assert not np.array_equal(nxt, sh.indices(0, learner))
    # deterministic, and uniform over positions (first slot over many epochs)
    a = mlp.Shuffler(5, 640, 4, 32).indices(7, 1)
    assert np.array_equal(a, mlp.Shuffler(5, 640, 4, 32).indices(7, 1))
    sh2 = mlp.Shuffler(9, 8, 1, 2)
    counts = np.zeros(8)
    for e in range(2000):
        counts[sh2.indices(4 * e, 0)[0, 0]] += 1
    chi2 = ((counts - 250.0) ** 2 / 250.0).sum()
    assert chi2 < 24.3  # p ~ 0.001 at 7 degrees of freedom
