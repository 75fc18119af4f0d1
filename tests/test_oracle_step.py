"""Pins for the oracle's step: closed forms, invariants and special cases that
reduce to a library routine (PyTorch's SGD with momentum)."""

import itertools

import numpy as np
import pytest
import torch

from oracle import mixing, step
from oracle.step import MIX_THEN_STEP, STEP_THEN_MIX


def _inputs(n, m, P, seed=0):
    rng = np.random.default_rng(seed)
    X = rng.standard_normal((n, P))
    V = rng.standard_normal((n, P)) * 0.1
    G = rng.standard_normal((n, m, P)) * 0.03
    return X, V, G


def _random_prefix_mask(rng, n, m):
    c = rng.integers(1, m + 1, size=n)
    return (np.arange(m)[None, :] < c[:, None]).astype(np.uint8)


def test_accumulate_special_cases():
    X, V, G = _inputs(3, 4, 5)
    full = np.ones((3, 4), np.uint8)
    np.testing.assert_allclose(step.accumulate(G, full), G.mean(axis=1), atol=1e-15)
    first = np.zeros((3, 4), np.uint8)
    first[:, 0] = 1
    np.testing.assert_array_equal(step.accumulate(G, first), G[:, 0])
    with pytest.raises(ValueError):
        step.accumulate(G, np.zeros((3, 4), np.uint8))


@pytest.mark.parametrize("order", [MIX_THEN_STEP, STEP_THEN_MIX])
def test_identity_w_no_momentum_is_lr_over_m_times_sum(order):
    # W = I, mu = 0: x_i' = x_i - (lr / m) * sum over finished j of G[i, j],
    # for any (also non-prefix) mask; linear in the finished count (Sec. 5.1).
    n, m, P = 3, 5, 7
    X, V, G = _inputs(n, m, P, 1)
    rng = np.random.default_rng(2)
    for _ in range(10):
        mask = (rng.random((n, m)) < 0.6).astype(np.uint8)
        mask[:, 2] = 1
        Xn, Vn = step.step(X, V, G, mask, np.eye(n), 0.3, 0.0, order)
        expect = X - (0.3 / m) * np.einsum("ij,ijp->ip", mask.astype(float), G)
        np.testing.assert_allclose(Xn, expect, rtol=0, atol=1e-14)
        # mu = 0: the buffer is just the finished-mini-batch mean
        cnt = mask.sum(axis=1)
        np.testing.assert_allclose(Vn * cnt[:, None], np.einsum("ij,ijp->ip", mask.astype(float), G),
                                   atol=1e-14)


@pytest.mark.parametrize("order", [MIX_THEN_STEP, STEP_THEN_MIX])
def test_permutation_w_moves_replicas_and_leaves_momentum(order):
    # A permutation matrix is doubly stochastic; W[i, p] = 1 puts replica p in
    # slot i.  Momentum buffers are never mixed.
    n, m, P = 4, 3, 6
    X, V, G = _inputs(n, m, P, 3)
    sigma = [2, 0, 3, 1]
    W = np.zeros((n, n))
    for i, p in enumerate(sigma):
        W[i, p] = 1.0
    mask = np.ones((n, m), np.uint8)
    mask[1, 2] = 0
    Xn, Vn = step.step(X, V, G, mask, W, 0.1, 0.9, order)
    Xi, Vi = step.step(X, V, G, mask, np.eye(n), 0.1, 0.9, order)
    np.testing.assert_array_equal(Vn, Vi)
    cnt = mask.sum(axis=1)
    eta = 0.1 * cnt / m
    for i, p in enumerate(sigma):
        if order == STEP_THEN_MIX:
            np.testing.assert_allclose(Xn[i], Xi[p], atol=1e-15)
        else:
            np.testing.assert_allclose(Xn[i], X[p] - eta[i] * Vn[i], atol=1e-15)


@pytest.mark.parametrize("order", [MIX_THEN_STEP, STEP_THEN_MIX])
def test_mean_preserved_by_any_doubly_stochastic_w(order):
    n, m, P = 8, 4, 9
    X, V, G = _inputs(n, m, P, 4)
    rng = np.random.default_rng(5)
    mask = _random_prefix_mask(rng, n, m)
    cnt = mask.sum(axis=1)
    for W in (mixing.w_ring(n), mixing.w_uniform(n), mixing.Matcha(1, n, 3).w(0)):
        Xn, Vn = step.step(X, V, G, mask, W, 0.2, 0.9, order)
        eta = 0.2 * cnt / m
        np.testing.assert_allclose(Xn.mean(axis=0), (X - eta[:, None] * Vn).mean(axis=0),
                                   atol=1e-14)


def test_uniform_mix_then_step_rows_differ_by_local_step():
    n, m, P = 4, 4, 5
    X, V, G = _inputs(n, m, P, 6)
    mask = _random_prefix_mask(np.random.default_rng(7), n, m)
    Xn, Vn = step.step(X, V, G, mask, mixing.w_uniform(n), 0.1, 0.9, MIX_THEN_STEP)
    eta = 0.1 * mask.sum(axis=1) / m
    base = Xn + eta[:, None] * Vn
    np.testing.assert_allclose(base, np.broadcast_to(X.mean(axis=0), base.shape), atol=1e-14)


def test_full_mask_allreduce_is_synchronous_sgd_with_momentum():
    # STEP_THEN_MIX with W = J/n and every mini-batch finished: after each step
    # all replicas are identical and equal to synchronous mini-batch SGD with
    # heavy-ball momentum (Eq. 2) on the mean gradient and the mean buffer.
    # Reference: torch.optim.SGD on one model, fp64 on the CPU.
    n, m, P, K = 4, 3, 6, 5
    rng = np.random.default_rng(8)
    X = rng.standard_normal((n, P))
    V = np.zeros((n, P))
    Gs = [rng.standard_normal((n, m, P)) * 0.05 for _ in range(K)]
    lr, mu = 0.1, 0.9
    W = mixing.w_uniform(n)
    mask = np.ones((n, m), np.uint8)
    x = torch.tensor(X.mean(axis=0), dtype=torch.float64, requires_grad=True)
    opt = torch.optim.SGD([x], lr=lr, momentum=mu)
    for k in range(K):
        X, V = step.step(X, V, Gs[k], mask, W, lr, mu, STEP_THEN_MIX)
        x.grad = torch.tensor(Gs[k].mean(axis=(0, 1)), dtype=torch.float64)
        opt.step()
        np.testing.assert_allclose(X, np.broadcast_to(X[0], X.shape), rtol=0, atol=1e-15)
        np.testing.assert_allclose(X[0], x.detach().numpy(), rtol=0, atol=1e-13)


def test_identity_w_each_learner_is_pytorch_sgd():
    # W = I decouples the learners: each one is torch SGD with momentum whose
    # learning rate is lr * c_i / m and whose gradient is its finished mean.
    n, m, P = 3, 4, 5
    rng = np.random.default_rng(9)
    X = rng.standard_normal((n, P))
    V = np.zeros((n, P))
    xs = [torch.tensor(X[i], dtype=torch.float64, requires_grad=True) for i in range(n)]
    opts = [torch.optim.SGD([x], lr=0.1, momentum=0.9) for x in xs]
    for k in range(4):
        G = rng.standard_normal((n, m, P))
        mask = _random_prefix_mask(rng, n, m)
        X, V = step.step(X, V, G, mask, np.eye(n), 0.1, 0.9, MIX_THEN_STEP)
        for i in range(n):
            c = int(mask[i].sum())
            for grp in opts[i].param_groups:
                grp["lr"] = 0.1 * c / m
            xs[i].grad = torch.tensor(G[i, :c].mean(axis=0), dtype=torch.float64)
            opts[i].step()
            np.testing.assert_allclose(X[i], xs[i].detach().numpy(), rtol=0, atol=1e-14)


def test_brute_force_all_masks_tiny():
    # every mask with at least one finished mini-batch per learner, n = 2,
    # m = 2, against a scalar per-element evaluation of the iteration
    n, m, P = 2, 2, 3
    X, V, G = _inputs(n, m, P, 10)
    W = np.array([[0.75, 0.25], [0.25, 0.75]])
    rows = [r for r in itertools.product([0, 1], repeat=m) if any(r)]
    for r0, r1 in itertools.product(rows, rows):
        mask = np.array([r0, r1], np.uint8)
        for order in (MIX_THEN_STEP, STEP_THEN_MIX):
            Xn, Vn = step.step(X, V, G, mask, W, 0.5, 0.5, order)
            for e in range(P):
                v = []
                for i in range(n):
                    done = [j for j in range(m) if mask[i, j]]
                    g = sum(G[i, j, e] for j in done) / len(done)
                    v.append(0.5 * V[i, e] + g)
                eta = [0.5 * mask[i].sum() / m for i in range(n)]
                for i in range(n):
                    if order == MIX_THEN_STEP:
                        x = sum(W[i, p] * X[p, e] for p in range(n)) - eta[i] * v[i]
                    else:
                        x = sum(W[i, p] * (X[p, e] - eta[p] * v[p]) for p in range(n))
                    assert Xn[i, e] == pytest.approx(x, abs=1e-14)
                    assert Vn[i, e] == pytest.approx(v[i], abs=1e-15)


def test_parameter_server_equals_uniform_step_then_mix_from_identical_replicas():
    # Alg. 3 (with 1/n) is the uniform-W step-then-mix iteration when every
    # learner starts from the server model: x' = mean_i (x - eta_i v_i').
    n, m, P = 5, 4, 7
    rng = np.random.default_rng(11)
    x = rng.standard_normal(P)
    V = rng.standard_normal((n, P)) * 0.1
    G = rng.standard_normal((n, m, P)) * 0.05
    mask = _random_prefix_mask(rng, n, m)
    xp, Vp = step.parameter_server_step(x, V, G, mask, 0.3, 0.8)
    Xs, Vs = step.step(np.tile(x, (n, 1)), V, G, mask, mixing.w_uniform(n), 0.3, 0.8, STEP_THEN_MIX)
    np.testing.assert_allclose(Xs, np.broadcast_to(xp, Xs.shape), atol=1e-14)
    np.testing.assert_array_equal(Vp, Vs)
    # one learner, no momentum: plain SGD with the finished-fraction rate
    x1, _ = step.parameter_server_step(x, np.zeros((1, P)), G[:1], mask[:1], 0.3, 0.0)
    c = int(mask[0].sum())
    np.testing.assert_allclose(x1, x - 0.3 * (c / m) * G[0, :c].mean(axis=0), atol=1e-15)
