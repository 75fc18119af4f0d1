"""Pins for the mixing matrices: double stochasticity, mean preservation, exact
structure of the ring and of MATCHA's graph, matchings and activations."""

import numpy as np
import pytest

from oracle import mixing


def _doubly_stochastic(W):
    assert (W >= 0).all()
    np.testing.assert_allclose(W.sum(axis=0), 1.0, atol=1e-12)
    np.testing.assert_allclose(W.sum(axis=1), 1.0, atol=1e-12)


@pytest.mark.parametrize("n", [1, 2, 3, 4, 8, 16])
def test_uniform_and_ring(n):
    for W in (mixing.w_uniform(n), mixing.w_ring(n)):
        _doubly_stochastic(W)
        assert np.array_equal(W, W.T)
    R = mixing.w_ring(n)
    if n >= 3:
        for i in range(n):
            nz = sorted(np.flatnonzero(R[i]).tolist())
            assert nz == sorted({(i - 1) % n, i, (i + 1) % n})
            assert (R[i][nz] == 1.0 / 3.0).all()


def test_ring_of_three_is_uniform():
    np.testing.assert_allclose(mixing.w_ring(3), mixing.w_uniform(3), rtol=0, atol=1e-16)


def test_mean_preserved_and_uniform_averages():
    rng = np.random.default_rng(0)
    Z = rng.standard_normal((8, 33))
    for W in (mixing.w_ring(8), mixing.w_uniform(8), mixing.Matcha(0, 8, 3).w(1)):
        np.testing.assert_allclose((W @ Z).mean(axis=0), Z.mean(axis=0), atol=1e-13)
    U = mixing.w_uniform(8) @ Z
    np.testing.assert_allclose(U, np.broadcast_to(Z.mean(axis=0), Z.shape), atol=1e-13)


def test_matcha_graph_and_matchings():
    g = mixing.Matcha(0, 16, 3)
    n = 16
    deg = np.zeros(n, dtype=int)
    seen = set()
    for u, v in g.edges:
        assert 0 <= u < v < n
        assert (u, v) not in seen
        seen.add((u, v))
        deg[u] += 1
        deg[v] += 1
    assert (deg == 3).all() and len(g.edges) == 24
    # connected (independent check via powers of the adjacency matrix)
    A = np.zeros((n, n))
    for u, v in g.edges:
        A[u, v] = A[v, u] = 1
    reach = np.linalg.matrix_power(A + np.eye(n), n)
    assert (reach > 0).all()
    # matchings partition the edges, each is a matching, at most 2*3-1 colours
    assert 3 <= g.num_matchings <= 5
    covered = []
    for q in range(g.num_matchings):
        mq = g.matching(q)
        nodes = [x for e in mq for x in e]
        assert len(nodes) == len(set(nodes))
        covered += mq
    assert sorted(covered) == g.edges


def test_matcha_w_structure():
    g = mixing.Matcha(0, 16, 3)
    assert g.alpha == 0.25
    saw_partial = False
    for step in range(50):
        W = g.w(step)
        _doubly_stochastic(W)
        assert np.array_equal(W, W.T)
        assert np.array_equal(W * 4, np.round(W * 4))  # multiples of 1/4: exact
        act = g.active(step)
        active_edges = {e for q, on in enumerate(act) if on for e in g.matching(q)}
        for i in range(16):
            for p in range(16):
                if i != p:
                    expect = 0.25 if (min(i, p), max(i, p)) in active_edges else 0.0
                    assert W[i, p] == expect
        saw_partial |= 0 < sum(act) < len(act)
    assert saw_partial


def test_matcha_activation_rate_and_all_off():
    g = mixing.Matcha(0, 16, 3)
    on = [a for s in range(2000) for a in g.active(s)]
    frac = np.mean(on)
    assert abs(frac - 0.5) < 4 * 0.5 / np.sqrt(len(on))
    # a step where nothing is active gives W = I
    for s in range(2000):
        if not any(g.active(s)):
            assert np.array_equal(g.w(s), np.eye(16))
            break
    else:
        pytest.fail("no all-inactive step in 2000 draws")


def test_graph_rejects_impossible():
    with pytest.raises(ValueError):
        mixing.random_regular_graph(0, 5, 3)  # odd number of half-edges


# ------------------------------------------------ MATCHA's own p and alpha
def _graph_laplacian(n, edges):
    # D - A from the adjacency matrix, built apart from the oracle's helper
    A = np.zeros((n, n))
    for u, v in edges:
        A[u, v] = A[v, u] = 1.0
    return np.diag(A.sum(axis=1)) - A


def _enumerated_second_moment(g, p, alpha):
    # E[W^T W] by summing over all 2^M activation patterns with their
    # probabilities (independent matchings)
    n, M = g.n, g.num_matchings
    Ls = [_graph_laplacian(n, g.matching(q)) for q in range(M)]
    E = np.zeros((n, n))
    for bits in range(1 << M):
        on = [(bits >> q) & 1 for q in range(M)]
        prob = np.prod([p[q] if on[q] else 1 - p[q] for q in range(M)])
        W = np.eye(n) - alpha * sum((Ls[q] for q in range(M) if on[q]), np.zeros((n, n)))
        E += prob * (W.T @ W)
    return E


@pytest.mark.parametrize("n", [8, 10, 12])
def test_degree_two_graph_is_a_cycle_with_known_spectrum(n):
    # a connected 2-regular graph is a cycle: Laplacian eigenvalues
    # 2 - 2 cos(2 pi k / n); lambda_2 = 2 - 2 cos(2 pi / n), lambda_max = 4 (n even)
    g = mixing.Matcha(3, n, 2)
    lam2, grad = g.connectivity([1.0] * g.num_matchings)
    assert lam2 == pytest.approx(2 - 2 * np.cos(2 * np.pi / n), abs=1e-12)
    # the supergradient entries v^T L_q v add up to v^T L v = lambda_2
    assert grad.sum() == pytest.approx(lam2, abs=1e-12)
    # budget 1: every matching always on, W = I - alpha L deterministic; the
    # best constant edge weight is 2 / (lambda_2 + lambda_max), with
    # ||W^2 - J/n|| = ((lambda_max - lambda_2) / (lambda_max + lambda_2))^2
    lam, rho = g.optimize(1.0, iterations=50)
    assert g.probs == [1.0] * g.num_matchings
    assert lam == pytest.approx(lam2, abs=1e-12)
    assert g.alpha == pytest.approx(2 / (lam2 + 4), rel=1e-7)
    assert rho == pytest.approx(((4 - lam2) / (4 + lam2)) ** 2, rel=1e-9)


@pytest.mark.parametrize("seed,n,degree", [(0, 8, 3), (1, 10, 4), (2, 6, 2)])
def test_second_moment_closed_form_equals_enumeration(seed, n, degree):
    g = mixing.Matcha(seed, n, degree)
    rng = np.random.default_rng(seed)
    for _ in range(3):
        p = rng.random(g.num_matchings)
        alpha = rng.random() / degree
        np.testing.assert_allclose(g.second_moment(p, alpha), _enumerated_second_moment(g, p, alpha),
                                   rtol=0, atol=1e-13)
        M = _enumerated_second_moment(g, p, alpha) - np.full((n, n), 1.0 / n)
        assert g.spectral(p, alpha) == pytest.approx(np.abs(np.linalg.eigvals(M)).max(), abs=1e-12)


def test_expected_laplacian_and_supergradient():
    g = mixing.Matcha(0, 16, 3)
    rng = np.random.default_rng(1)
    p = rng.random(g.num_matchings)
    Lb = sum(p[q] * _graph_laplacian(16, g.matching(q)) for q in range(g.num_matchings))
    np.testing.assert_allclose(g.expected_laplacian(p), Lb, atol=1e-15)
    lam, grad = g.connectivity(p)
    assert lam == pytest.approx(np.sort(np.linalg.eigvals(Lb).real)[1], abs=1e-12)
    # lambda_2 is concave in p and, where simple, differentiable with gradient
    # v^T L_q v: central differences agree
    for q in range(g.num_matchings):
        h = 1e-6
        e = np.zeros_like(p)
        e[q] = h
        fd = (g.connectivity(p + e)[0] - g.connectivity(p - e)[0]) / (2 * h)
        assert grad[q] == pytest.approx(fd, abs=1e-6)


def test_projection_onto_capped_simplex():
    rng = np.random.default_rng(2)
    for _ in range(50):
        y = rng.normal(0.5, 0.8, size=6)
        total = rng.uniform(0.5, 5.0)
        x = mixing._project_capped(y, total)
        assert (x >= 0).all() and (x <= 1).all() and x.sum() <= total + 1e-9
        # optimality: no feasible point from a random sample is closer to y
        for _ in range(200):
            z = np.clip(rng.random(6), 0, 1)
            if z.sum() > total:
                z *= total / z.sum()
            assert np.linalg.norm(x - y) <= np.linalg.norm(z - y) + 1e-9


@pytest.mark.parametrize("seed,n,degree,budget", [(0, 8, 3, 0.5), (4, 8, 3, 0.3), (1, 10, 4, 0.5)])
def test_optimized_probabilities_beat_a_feasible_grid(seed, n, degree, budget):
    g = mixing.Matcha(seed, n, degree)
    M = g.num_matchings
    lam, rho = g.optimize(budget, iterations=1500)
    p = np.array(g.probs)
    assert (p >= 0).all() and (p <= 1).all() and p.sum() <= budget * M + 1e-9
    # brute force: lambda_2 over every grid point (step 0.1) of the feasible set
    Ls = np.stack([_graph_laplacian(n, g.matching(q)) for q in range(M)])
    grid = np.stack(np.meshgrid(*[np.linspace(0, 1, 11)] * M, indexing="ij"), -1).reshape(-1, M)
    grid = grid[grid.sum(axis=1) <= budget * M + 1e-12]
    lam_grid = np.linalg.eigvalsh(np.einsum("kq,qij->kij", grid, Ls))[:, 1].max()
    assert lam >= lam_grid - 1e-3
    assert lam == pytest.approx(np.linalg.eigvalsh(np.einsum("q,qij->ij", p, Ls))[1], abs=1e-12)
    # alpha: no point of a fine grid over (0, 1/degree] does better (exact E[W^T W])
    # E[W^T W] = I - 2 a E[L_S] + a^2 E[L_S^2] over the active set S: both
    # moments by enumeration, then every grid alpha at once
    J = np.full((n, n), 1.0 / n)
    E1 = (_enumerated_second_moment(g, p, -1.0) - _enumerated_second_moment(g, p, 1.0)) / 4
    E2 = (_enumerated_second_moment(g, p, 1.0) + _enumerated_second_moment(g, p, -1.0)) / 2 - np.eye(n)
    alphas = np.linspace(1e-4, 1.0 / degree, 3000)
    mats = np.eye(n) - 2 * alphas[:, None, None] * E1 + alphas[:, None, None] ** 2 * E2 - J
    best = np.abs(np.linalg.eigvalsh(mats)).max(axis=1).min()
    np.testing.assert_allclose(mats[1234] + J, _enumerated_second_moment(g, p, alphas[1234]), atol=1e-13)
    assert rho <= best + 1e-9
    assert 0 < g.alpha <= 1.0 / degree
    # the budget binds: the expected number of active matchings is at most b * M
    # and raising p anywhere (a bigger budget) cannot lower lambda_2
    lam_more, _ = mixing.Matcha(seed, n, degree).optimize(min(1.0, budget + 0.2), iterations=1500)
    assert lam_more >= lam - 1e-3


def test_optimized_activation_rate_and_sampled_second_moment():
    g = mixing.Matcha(0, 8, 3)
    g.optimize(0.5, iterations=600)
    steps = 4000
    on = np.array([g.active(s) for s in range(steps)], dtype=float)
    p = np.array(g.probs)
    se = np.sqrt(p * (1 - p) / steps)
    assert (np.abs(on.mean(axis=0) - p) <= 4 * se + 1e-12).all()
    Ws = [g.w(s) for s in range(steps)]
    emp = sum(W.T @ W for W in Ws) / steps
    assert np.abs(emp - g.second_moment(p, g.alpha)).max() < 0.03
