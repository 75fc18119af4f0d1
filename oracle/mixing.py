"""Mixing matrices W (x_i <- sum_p W[i, p] x_p; Alg. 2 averaging step, Eq. 6).

* uniform:  W = J / n, every entry 1/n.  Ring all-reduce averages all models
            (Eq. 4-5), which is this W.
* ring:     D-PSGD on a ring: each learner averages itself and its two ring
            neighbours with weight 1/3 (W = (I + S + S^T) / 3, S the cyclic
            shift).  n = 2 has one neighbour (weights 1/2); n = 1 is [1].
* MATCHA:   the base graph (a random d-regular simple connected graph, drawn by
            the pairing model) is split into matchings by greedy edge colouring;
            at every iteration matching q is active with probability p_q and
            W = I - alpha * sum_{active q} L_q with L_q the Laplacian of matching
            q.  Default p_q = 1/2 (communication budget 0.5, Sec. 6.1) and
            alpha = 1 / (max degree + 1); ``Matcha.optimize`` makes MATCHA's own
            choice instead (p maximising the algebraic connectivity of the
            expected graph under the budget, alpha minimising the spectral norm
            of E[W^T W] - J/n).

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
    if degree == 1 and n > 2:
        raise ValueError("a 1-regular graph (a perfect matching) is connected only on 2 nodes")
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


def matching_active(seed: int, step: int, q: int, p: float = 0.5) -> bool:
    """Matching q takes part in iteration ``step`` with probability p: u < p
    for u from Philox word 0 at counter (step, q, 0, 0) under key (seed, 3).
    (For p = 1/2 this is: the word's top bit is 0.)"""
    return philox.u01(philox.word(seed, philox.PURPOSE_ACTIVATION, step, q)) < p


def _project_capped(y, total):
    """Euclidean projection onto {0 <= p_q <= 1, sum p_q <= total}.  By the
    KKT conditions the projection is clip(y - tau, 0, 1) with tau >= 0 the
    smallest shift that meets the budget: tau = 0 if clip(y, 0, 1) already
    does, else the root of sum clip(y - tau, 0, 1) = total (bisection; the sum
    is non-increasing in tau)."""
    y = np.asarray(y, dtype=np.float64)
    p = np.clip(y, 0.0, 1.0)
    if p.sum() <= total:
        return p
    lo, hi = 0.0, float(y.max())
    for _ in range(200):
        tau = 0.5 * (lo + hi)
        if np.clip(y - tau, 0.0, 1.0).sum() > total:
            lo = tau
        else:
            hi = tau
    return np.clip(y - hi, 0.0, 1.0)


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
        self.probs = [0.5] * self.num_matchings

    def matching(self, q: int):
        return [e for e, c in zip(self.edges, self.colours) if c == q]

    def active(self, step: int):
        return [matching_active(self.seed, step, q, self.probs[q]) for q in range(self.num_matchings)]

    # ---------------------------------------------- MATCHA's own p and alpha
    def expected_laplacian(self, p) -> np.ndarray:
        return sum(p[q] * laplacian(self.n, self.matching(q)) for q in range(self.num_matchings))

    def connectivity(self, p):
        """(lambda_2 of the expected Laplacian, its supergradient v^T L_q v)."""
        w, V = np.linalg.eigh(self.expected_laplacian(p))
        v = V[:, 1]
        grad = np.array([sum((v[a] - v[b]) ** 2 for a, b in self.matching(q))
                         for q in range(self.num_matchings)])
        return float(w[1]), grad

    def second_moment(self, p, alpha) -> np.ndarray:
        """E[W^T W] for independent activations, in closed form:
        I - 2 alpha Lbar + alpha^2 (Lbar^2 + sum_q p_q (1 - p_q) L_q^2)."""
        Lb = self.expected_laplacian(p)
        var = sum(p[q] * (1 - p[q]) * np.linalg.matrix_power(laplacian(self.n, self.matching(q)), 2)
                  for q in range(self.num_matchings))
        return np.eye(self.n) - 2 * alpha * Lb + alpha ** 2 * (Lb @ Lb + var)

    def spectral(self, p, alpha) -> float:
        M = self.second_moment(p, alpha) - np.full((self.n, self.n), 1.0 / self.n)
        return float(np.max(np.abs(np.linalg.eigvalsh(M))))

    def optimize(self, budget: float, iterations: int = 2000):
        """p: projected supergradient ascent of lambda_2 on {0 <= p <= 1,
        sum p <= budget * M} (step 0.5 / sqrt(k + 1) along the normalised
        supergradient, the best iterate kept); alpha: the minimiser of
        ``spectral`` over (0, 1/degree] (400-point grid, then golden section).
        Returns (lambda_2, spectral norm)."""
        M = self.num_matchings
        total = budget * M
        p = np.full(M, min(1.0, budget))
        best, best_val = p.copy(), self.connectivity(p)[0]
        for k in range(iterations):
            _, g = self.connectivity(p)
            gn = np.linalg.norm(g)
            if gn == 0:
                break
            p = _project_capped(p + (0.5 / np.sqrt(k + 1.0)) * g / gn, total)
            val = self.connectivity(p)[0]
            if val > best_val:
                best, best_val = p.copy(), val
        hi = 1.0 / self.degree
        grid = [hi * k / 400.0 for k in range(1, 401)]
        vals = [self.spectral(best, a) for a in grid]
        a_best = grid[int(np.argmin(vals))]
        lo, up = max(0.0, a_best - hi / 400.0), min(hi, a_best + hi / 400.0)
        phi = 0.5 * (np.sqrt(5.0) - 1.0)
        for _ in range(60):
            x1, x2 = up - phi * (up - lo), lo + phi * (up - lo)
            if self.spectral(best, x1) < self.spectral(best, x2):
                up = x2
            else:
                lo = x1
        a_ref = 0.5 * (lo + up)
        if self.spectral(best, a_ref) < min(vals):
            a_best = a_ref
        self.probs = [float(x) for x in best]
        self.alpha = float(a_best)
        return best_val, self.spectral(best, a_best)

    def w(self, step: int) -> np.ndarray:
        W = np.eye(self.n, dtype=np.float64)
        for q, on in enumerate(self.active(step)):
            if on:
                W = W - self.alpha * laplacian(self.n, self.matching(q))
        return W
