"""Mixing matrices W (x_i <- sum_p W[i, p] x_p; Alg. 2 averaging step, Eq. 6).

* uniform:  W = J / n, every entry 1/n.  Ring all-reduce averages all models
            (Eq. 4-5), which is this W.
* ring:     D-PSGD on a ring: each learner averages itself and its two ring
            neighbours with weight 1/3 (W = (I + S + S^T) / 3, S the cyclic
            shift).  n = 2 has one neighbour (weights 1/2); n = 1 is [1].
* MATCHA:   the base graph (a random d-regular simple connected graph, drawn by
            the pairing model) is split into matchings by greedy edge colouring;
            at every iteration each matching is active with probability 1/2
            (communication budget 0.5, Sec. 6.1) and
            W = I - alpha * sum_{active q} L_q with L_q the Laplacian of matching
            q and alpha = 1 / (max degree + 1).

All builders return fp64 matrices; every W here is symmetric and doubly
stochastic with non-negative entries.
"""

from __future__ import annotations

import numpy as np

from . import philox


def w_uniform(n: int) -> np.ndarray:
    return np.full((n, n), 1.0 / n, dtype=np.float64)


def w_ring(n: int) -> np.ndarray:
    if n == 1:
        return np.ones((1, 1), dtype=np.float64)
    if n == 2:
        return np.full((2, 2), 0.5, dtype=np.float64)
    W = np.zeros((n, n), dtype=np.float64)
    for i in range(n):
        for p in (i - 1, i, i + 1):
            W[i, p % n] = 1.0 / 3.0
    return W


def _connected(n: int, edges) -> bool:
    adj = [[] for _ in range(n)]
    for u, v in edges:
        adj[u].append(v)
        adj[v].append(u)
    seen = {0}
    todo = [0]
    while todo:
        u = todo.pop()
        for v in adj[u]:
            if v not in seen:
                seen.add(v)
                todo.append(v)
    return len(seen) == n


def random_regular_graph(seed: int, n: int, degree: int, max_attempts: int = 100000):
    """Random ``degree``-regular simple connected graph on n nodes (pairing model).

    Half-edges 0 .. n*degree-1 belong to node h // degree.  Attempt a shuffles
    them with Fisher-Yates from the top (position t swaps with a uniform
    position r in [0, t], r from Philox word 0 at counter (a, t, 0, 0) under key
    (seed, 2)) and pairs consecutive half-edges.  A result with a self-loop, a
    repeated edge or more than one component is rejected and the next attempt
    is drawn.  Returns (edges sorted with u < v, attempts used).
    """
    if n < 2 or degree < 1 or degree >= n or (n * degree) % 2:
        raise ValueError("no simple regular graph with these n and degree")
    H = n * degree
    for attempt in range(max_attempts):
        half = list(range(H))
        for t in range(H - 1, 0, -1):
            r = philox.bounded(philox.word(seed, philox.PURPOSE_GRAPH, attempt, t), t + 1)
            half[t], half[r] = half[r], half[t]
        edges = set()
        ok = True
        for k in range(0, H, 2):
            u, v = half[k] // degree, half[k + 1] // degree
            if u == v:
                ok = False
                break
            e = (min(u, v), max(u, v))
            if e in edges:
                ok = False
                break
            edges.add(e)
        if ok and _connected(n, edges):
            return sorted(edges), attempt + 1
    raise RuntimeError("pairing model did not produce a simple connected graph")


def greedy_matchings(edges):
    """Split edges into matchings: in lexicographic order, each edge takes the
    smallest colour not yet used by an edge at either endpoint.  Returns the
    list of colours (aligned with ``edges``) and the number of matchings."""
    used = {}
    colours = []
    for u, v in sorted(edges):
        taken = used.get(u, set()) | used.get(v, set())
        c = 0
        while c in taken:
            c += 1
        colours.append(c)
        used.setdefault(u, set()).add(c)
        used.setdefault(v, set()).add(c)
    return colours, (max(colours) + 1 if colours else 0)


def matching_active(seed: int, step: int, q: int) -> bool:
    """Matching q takes part in iteration ``step`` with probability 1/2: the top
    bit of Philox word 0 at counter (step, q, 0, 0) under key (seed, 3) is 0."""
    return (philox.word(seed, philox.PURPOSE_ACTIVATION, step, q) >> 63) == 0


def laplacian(n: int, edges) -> np.ndarray:
    L = np.zeros((n, n), dtype=np.float64)
    for u, v in edges:
        L[u, u] += 1.0
        L[v, v] += 1.0
        L[u, v] -= 1.0
        L[v, u] -= 1.0
    return L


class Matcha:
    """MATCHA state: a fixed base graph and its matchings; W changes per step."""

    def __init__(self, seed: int, n: int, degree: int):
        self.seed, self.n, self.degree = seed, n, degree
        self.edges, self.attempts = random_regular_graph(seed, n, degree)
        self.colours, self.num_matchings = greedy_matchings(self.edges)
        self.alpha = 1.0 / (degree + 1)

    def matching(self, q: int):
        return [e for e, c in zip(self.edges, self.colours) if c == q]

    def active(self, step: int):
        return [matching_active(self.seed, step, q) for q in range(self.num_matchings)]

    def w(self, step: int) -> np.ndarray:
        W = np.eye(self.n, dtype=np.float64)
        for q, on in enumerate(self.active(step)):
            if on:
                W = W - self.alpha * laplacian(self.n, self.matching(q))
        return W
