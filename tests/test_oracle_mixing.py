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
