// MATCHA mixing (the decentralized baseline the paper runs with a
// communication budget, Sec. 6.1): a random regular base graph split into
// matchings, each matching active at an iteration with its own probability,
// and W = I - alpha * sum of the active matchings' Laplacians.
//
// Default: every matching active with probability 1/2 (budget 0.5 spread
// evenly) and alpha = 1 / (degree + 1).  nbsgd_matcha_optimize replaces both
// by MATCHA's own choice: probabilities that maximise the algebraic
// connectivity of the expected graph under the budget, and the alpha that
// minimises the spectral norm of E[W^T W] - J/n.
#include <math.h>

#include <algorithm>
#include <new>
#include <set>
#include <utility>
#include <vector>

#include "internal.h"

using namespace nbsgd;

struct nbsgd_matcha {
  uint64_t seed;
  int32_t n, degree, matchings;
  double alpha;
  std::vector<std::pair<int32_t, int32_t>> edges;  // u < v, lexicographic
  std::vector<int32_t> colour;                     // matching of each edge
  std::vector<double> prob;                        // activation probability per matching
};

namespace {

bool connected(int32_t n, const std::vector<std::pair<int32_t, int32_t>>& edges) {
  std::vector<std::vector<int32_t>> adj(n);
  for (auto& e : edges) {
    adj[e.first].push_back(e.second);
    adj[e.second].push_back(e.first);
  }
  std::vector<char> seen(n, 0);
  std::vector<int32_t> todo{0};
  seen[0] = 1;
  int32_t reached = 1;
  while (!todo.empty()) {
    const int32_t u = todo.back();
    todo.pop_back();
    for (int32_t v : adj[u])
      if (!seen[v]) {
        seen[v] = 1;
        ++reached;
        todo.push_back(v);
      }
  }
  return reached == n;
}

// ---- small dense symmetric algebra (n <= 16) --------------------------------
using Mat = std::vector<double>;  // row-major n x n

// Eigen-decomposition of a symmetric matrix by cyclic Jacobi rotations: each
// rotation zeroes one off-diagonal pair; sweeps repeat until the off-diagonal
// mass is negligible.  Returns eigenvalues ascending, eigenvectors as columns.
void sym_eig(int n, Mat a, std::vector<double>& evals, Mat& vecs) {
  vecs.assign((size_t)n * n, 0.0);
  for (int i = 0; i < n; ++i) vecs[(size_t)i * n + i] = 1.0;
  for (int sweep = 0; sweep < 100; ++sweep) {
    double off = 0.0, total = 0.0;
    for (int i = 0; i < n; ++i)
      for (int j = 0; j < n; ++j) {
        total += a[(size_t)i * n + j] * a[(size_t)i * n + j];
        if (i != j) off += a[(size_t)i * n + j] * a[(size_t)i * n + j];
      }
    if (off <= 1e-30 * (total + 1e-300)) break;
    for (int p = 0; p < n - 1; ++p)
      for (int q = p + 1; q < n; ++q) {
        const double apq = a[(size_t)p * n + q];
        if (apq == 0.0) continue;
        const double theta = (a[(size_t)q * n + q] - a[(size_t)p * n + p]) / (2.0 * apq);
        const double t = (theta >= 0 ? 1.0 : -1.0) / (fabs(theta) + sqrt(theta * theta + 1.0));
        const double c = 1.0 / sqrt(t * t + 1.0), s = t * c;
        for (int k = 0; k < n; ++k) {  // columns p, q
          const double akp = a[(size_t)k * n + p], akq = a[(size_t)k * n + q];
          a[(size_t)k * n + p] = c * akp - s * akq;
          a[(size_t)k * n + q] = s * akp + c * akq;
        }
        for (int k = 0; k < n; ++k) {  // rows p, q
          const double apk = a[(size_t)p * n + k], aqk = a[(size_t)q * n + k];
          a[(size_t)p * n + k] = c * apk - s * aqk;
          a[(size_t)q * n + k] = s * apk + c * aqk;
        }
        for (int k = 0; k < n; ++k) {
          const double vkp = vecs[(size_t)k * n + p], vkq = vecs[(size_t)k * n + q];
          vecs[(size_t)k * n + p] = c * vkp - s * vkq;
          vecs[(size_t)k * n + q] = s * vkp + c * vkq;
        }
      }
  }
  std::vector<int> order(n);
  for (int i = 0; i < n; ++i) order[i] = i;
  std::sort(order.begin(), order.end(),
            [&](int x, int y) { return a[(size_t)x * n + x] < a[(size_t)y * n + y]; });
  evals.resize(n);
  Mat sorted((size_t)n * n);
  for (int k = 0; k < n; ++k) {
    evals[k] = a[(size_t)order[k] * n + order[k]];
    for (int i = 0; i < n; ++i) sorted[(size_t)i * n + k] = vecs[(size_t)i * n + order[k]];
  }
  vecs.swap(sorted);
}

// Expected Laplacian sum_q p_q L_q.
Mat expected_laplacian(const nbsgd_matcha& g, const std::vector<double>& p) {
  const int n = g.n;
  Mat L((size_t)n * n, 0.0);
  for (size_t k = 0; k < g.edges.size(); ++k) {
    const double w = p[g.colour[k]];
    const int u = g.edges[k].first, v = g.edges[k].second;
    L[(size_t)u * n + u] += w;
    L[(size_t)v * n + v] += w;
    L[(size_t)u * n + v] -= w;
    L[(size_t)v * n + u] -= w;
  }
  return L;
}

// lambda_2 of the expected Laplacian and a supergradient with respect to p:
// d lambda_2 / d p_q = v^T L_q v for the unit eigenvector v of lambda_2.
double fiedler(const nbsgd_matcha& g, const std::vector<double>& p, std::vector<double>* grad) {
  std::vector<double> ev;
  Mat vecs;
  sym_eig(g.n, expected_laplacian(g, p), ev, vecs);
  if (grad) {
    grad->assign(g.matchings, 0.0);
    for (size_t k = 0; k < g.edges.size(); ++k) {
      const double d = vecs[(size_t)g.edges[k].first * g.n + 1] - vecs[(size_t)g.edges[k].second * g.n + 1];
      (*grad)[g.colour[k]] += d * d;
    }
  }
  return ev[1];
}

// Euclidean projection onto {0 <= p_q <= 1, sum p_q <= budget}.
void project(std::vector<double>& p, double budget) {
  // Euclidean projection onto {0 <= p <= 1, sum p <= budget}: clip(y - tau)
  // with the smallest tau >= 0 that meets the budget (KKT conditions).
  const std::vector<double> y = p;
  double s = 0.0;
  for (double& x : p) {
    x = std::min(1.0, std::max(0.0, x));
    s += x;
  }
  if (s <= budget) return;
  double lo = 0.0, hi = *std::max_element(y.begin(), y.end());
  for (int it = 0; it < 200; ++it) {  // sum of clip(y - tau) is non-increasing in tau
    const double tau = 0.5 * (lo + hi);
    double t = 0.0;
    for (double x : y) t += std::min(1.0, std::max(0.0, x - tau));
    (t > budget ? lo : hi) = tau;
  }
  for (size_t q = 0; q < p.size(); ++q) p[q] = std::min(1.0, std::max(0.0, y[q] - hi));
}

// Spectral norm of E[W^T W] - J/n for W = I - alpha * sum_q B_q L_q with
// independent B_q ~ Bernoulli(p_q): E[W^T W] = I - 2 alpha Lbar + alpha^2
// (Lbar^2 + sum_q p_q (1 - p_q) L_q^2), and L_q^2 = 2 L_q for a matching.
double rho(const nbsgd_matcha& g, const std::vector<double>& p, double alpha) {
  const int n = g.n;
  const Mat Lb = expected_laplacian(g, p);
  std::vector<double> var(g.matchings);
  for (int q = 0; q < g.matchings; ++q) var[q] = 2.0 * p[q] * (1.0 - p[q]);
  const Mat Lv = expected_laplacian(g, var);
  Mat M((size_t)n * n);
  for (int i = 0; i < n; ++i)
    for (int j = 0; j < n; ++j) {
      double l2 = 0.0;
      for (int k = 0; k < n; ++k) l2 += Lb[(size_t)i * n + k] * Lb[(size_t)k * n + j];
      M[(size_t)i * n + j] = (i == j ? 1.0 : 0.0) - 1.0 / n - 2.0 * alpha * Lb[(size_t)i * n + j] +
                             alpha * alpha * (l2 + Lv[(size_t)i * n + j]);
    }
  std::vector<double> ev;
  Mat vecs;
  sym_eig(n, M, ev, vecs);
  return std::max(fabs(ev.front()), fabs(ev.back()));
}

}  // namespace

extern "C" nbsgd_status nbsgd_matcha_create(uint64_t seed, int32_t n, int32_t degree,
                                            nbsgd_matcha** out) {
  clear_error();
  if (!out) return fail(NBSGD_E_ARG, "out is null");
  *out = nullptr;
  if (nbsgd_status st = check_nm(n, 1)) return st;
  if (n < 2 || degree < 1 || degree >= n || (n * degree) % 2)
    return fail(NBSGD_E_SHAPE, "no simple %d-regular graph on %d nodes", degree, n);
  if (degree == 1 && n > 2)  // a perfect matching is connected only on two nodes
    return fail(NBSGD_E_SHAPE, "no connected 1-regular graph on %d nodes", n);
  const int32_t H = n * degree;
  std::vector<int32_t> half(H);
  std::vector<std::pair<int32_t, int32_t>> edges;
  bool found = false;
  for (uint64_t attempt = 0; attempt < 100000 && !found; ++attempt) {
    for (int32_t h = 0; h < H; ++h) half[h] = h;
    for (int32_t t = H - 1; t >= 1; --t) {
      const uint64_t r = below(draw(seed, kPurposeGraph, attempt, (uint64_t)t, 0), (uint64_t)t + 1);
      std::swap(half[t], half[r]);
    }
    std::set<std::pair<int32_t, int32_t>> es;
    bool ok = true;
    for (int32_t k = 0; k < H && ok; k += 2) {
      const int32_t u = half[k] / degree, v = half[k + 1] / degree;
      if (u == v) ok = false;
      else ok = es.insert({std::min(u, v), std::max(u, v)}).second;
    }
    if (!ok) continue;
    edges.assign(es.begin(), es.end());  // std::set orders lexicographically
    found = connected(n, edges);
  }
  if (!found) return fail(NBSGD_E_SHAPE, "pairing model found no connected simple graph");

  nbsgd_matcha* g = new (std::nothrow) nbsgd_matcha;
  if (!g) return fail(NBSGD_E_ARG, "out of host memory");
  g->seed = seed;
  g->n = n;
  g->degree = degree;
  g->alpha = 1.0 / (double)(degree + 1);
  g->edges = edges;
  g->colour.assign(edges.size(), 0);
  std::vector<std::set<int32_t>> used(n);
  int32_t M = 0;
  for (size_t k = 0; k < edges.size(); ++k) {
    const int32_t u = edges[k].first, v = edges[k].second;
    int32_t c = 0;
    while (used[u].count(c) || used[v].count(c)) ++c;
    g->colour[k] = c;
    used[u].insert(c);
    used[v].insert(c);
    M = std::max(M, c + 1);
  }
  g->matchings = M;
  g->prob.assign(M, 0.5);
  *out = g;
  return NBSGD_OK;
}

extern "C" nbsgd_status nbsgd_matcha_w(const nbsgd_matcha* g, uint64_t step, float* W,
                                       int32_t* n_active) {
  clear_error();
  if (!g || !W) return fail(NBSGD_E_ARG, "g and W must not be null");
  const int32_t n = g->n;
  std::vector<double> acc((size_t)n * n, 0.0);
  for (int32_t i = 0; i < n; ++i) acc[(size_t)i * n + i] = 1.0;
  int32_t active = 0;
  for (int32_t q = 0; q < g->matchings; ++q) {
    if (!(open_unit(draw(g->seed, kPurposeActivation, step, (uint64_t)q, 0)) < g->prob[q])) continue;
    ++active;
    for (size_t k = 0; k < g->edges.size(); ++k) {
      if (g->colour[k] != q) continue;
      const int32_t u = g->edges[k].first, v = g->edges[k].second;
      acc[(size_t)u * n + u] -= g->alpha;
      acc[(size_t)v * n + v] -= g->alpha;
      acc[(size_t)u * n + v] += g->alpha;
      acc[(size_t)v * n + u] += g->alpha;
    }
  }
  for (size_t k = 0; k < acc.size(); ++k) W[k] = (float)acc[k];
  if (n_active) *n_active = active;
  return NBSGD_OK;
}

extern "C" nbsgd_status nbsgd_matcha_matchings(const nbsgd_matcha* g, int32_t* edges_uvq,
                                               int32_t* E, int32_t* M) {
  clear_error();
  if (!g || !E || !M) return fail(NBSGD_E_ARG, "g, E and M must not be null");
  *E = (int32_t)g->edges.size();
  *M = g->matchings;
  if (edges_uvq)
    for (size_t k = 0; k < g->edges.size(); ++k) {
      edges_uvq[3 * k + 0] = g->edges[k].first;
      edges_uvq[3 * k + 1] = g->edges[k].second;
      edges_uvq[3 * k + 2] = g->colour[k];
    }
  return NBSGD_OK;
}

extern "C" nbsgd_status nbsgd_matcha_set(nbsgd_matcha* g, const double* probs, double alpha) {
  clear_error();
  if (!g || !probs) return fail(NBSGD_E_ARG, "g and probs must not be null");
  for (int32_t q = 0; q < g->matchings; ++q)
    if (!(probs[q] >= 0.0 && probs[q] <= 1.0))
      return fail(NBSGD_E_ARG, "probs[%d]=%g is outside [0, 1]", q, probs[q]);
  if (!(alpha > 0.0) || !(alpha * g->degree <= 1.0))
    return fail(NBSGD_E_ARG, "alpha=%g must be in (0, 1/degree] so W stays non-negative", alpha);
  g->prob.assign(probs, probs + g->matchings);
  g->alpha = alpha;
  return NBSGD_OK;
}

extern "C" nbsgd_status nbsgd_matcha_get(const nbsgd_matcha* g, double* probs, double* alpha) {
  clear_error();
  if (!g) return fail(NBSGD_E_ARG, "g is null");
  if (probs) std::copy(g->prob.begin(), g->prob.end(), probs);
  if (alpha) *alpha = g->alpha;
  return NBSGD_OK;
}

extern "C" nbsgd_status nbsgd_matcha_optimize(nbsgd_matcha* g, double budget, int32_t iterations,
                                              double* lambda2, double* spectral) {
  clear_error();
  if (!g) return fail(NBSGD_E_ARG, "g is null");
  if (!(budget > 0.0 && budget <= 1.0)) return fail(NBSGD_E_ARG, "budget %g must be in (0, 1]", budget);
  if (iterations < 1) return fail(NBSGD_E_ARG, "iterations must be >= 1");
  const int M = g->matchings;
  const double total = budget * M;
  // projected supergradient ascent on the concave lambda_2(sum_q p_q L_q)
  std::vector<double> p(M, std::min(1.0, budget)), grad, best = p;
  double best_val = fiedler(*g, p, nullptr);
  for (int k = 0; k < iterations; ++k) {
    fiedler(*g, p, &grad);
    double gn = 0.0;
    for (double x : grad) gn += x * x;
    gn = sqrt(gn);
    if (gn == 0.0) break;
    const double t = 0.5 / sqrt((double)k + 1.0);
    for (int q = 0; q < M; ++q) p[q] += t * grad[q] / gn;
    project(p, total);
    const double val = fiedler(*g, p, nullptr);
    if (val > best_val) {
      best_val = val;
      best = p;
    }
  }
  // alpha: grid over (0, 1/degree], then golden-section refinement
  const double hi = 1.0 / g->degree;
  double a_best = hi, r_best = rho(*g, best, hi);
  for (int k = 1; k <= 400; ++k) {
    const double a = hi * k / 400.0;
    const double r = rho(*g, best, a);
    if (r < r_best) {
      r_best = r;
      a_best = a;
    }
  }
  double lo = std::max(0.0, a_best - hi / 400.0), up = std::min(hi, a_best + hi / 400.0);
  const double phi = 0.5 * (sqrt(5.0) - 1.0);
  for (int it = 0; it < 60; ++it) {
    const double x1 = up - phi * (up - lo), x2 = lo + phi * (up - lo);
    if (rho(*g, best, x1) < rho(*g, best, x2))
      up = x2;
    else
      lo = x1;
  }
  const double a_ref = 0.5 * (lo + up);
  if (rho(*g, best, a_ref) < r_best) {
    a_best = a_ref;
    r_best = rho(*g, best, a_ref);
  }
  g->prob = best;
  g->alpha = a_best;
  if (lambda2) *lambda2 = best_val;
  if (spectral) *spectral = r_best;
  return NBSGD_OK;
}

extern "C" void nbsgd_matcha_destroy(nbsgd_matcha* g) { delete g; }
