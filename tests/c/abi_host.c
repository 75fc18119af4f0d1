/* The host entry points of libnbsgd called from plain C11 through
 * include/nbsgd.h: the iteration schedule, the mixing matrices, MATCHA, the
 * row stride, the MLP shape helpers, the local shuffle and their error paths.
 * No GPU is touched.  Prints "ok" and exits 0 when every check holds. */
#include <math.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "nbsgd.h"

static int failures = 0;

#define CHECK(cond)                                                   \
  do {                                                                \
    if (!(cond)) {                                                    \
      fprintf(stderr, "%s:%d: check failed: %s\n", __FILE__, __LINE__, #cond); \
      ++failures;                                                     \
    }                                                                 \
  } while (0)

static void doubly_stochastic(const float *W, int n) {
  for (int i = 0; i < n; ++i) {
    double row = 0.0, col = 0.0;
    for (int p = 0; p < n; ++p) {
      CHECK(W[i * n + p] >= 0.0f);
      row += W[i * n + p];
      col += W[p * n + i];
    }
    CHECK(fabs(row - 1.0) < 1e-6 && fabs(col - 1.0) < 1e-6);
  }
}

static void schedule(void) {
  enum { n = 8, m = 8 };
  uint8_t mask[n * m];
  int32_t counts[n];
  double times[n * m], timing[3];
  nbsgd_delay d = {NBSGD_DELAY_EXP, 1.0, 1.0, 7, 3.0, 0.0};
  for (uint64_t step = 0; step < 20; ++step) {
    CHECK(nbsgd_sample_mask(0, step, n, m, &d, mask, counts, times, timing) == NBSGD_OK);
    int full = 0;
    for (int i = 0; i < n; ++i) {
      CHECK(counts[i] >= 1 && counts[i] <= m);
      full |= counts[i] == m;
      for (int j = 0; j < m; ++j) CHECK(mask[i * m + j] == (j < counts[i]));
      /* learner 7 is slowed by 3 on every mini-batch, base 1 included */
      if (i == 7) CHECK(times[i * m] >= 3.0);
    }
    CHECK(full); /* the learner that sent the terminal signal finished all m */
    CHECK(timing[0] <= timing[2] && timing[2] <= timing[1]);
    /* Sec. 4.3 accounting: X_{1:P} and X_{P:P} are the two iteration times,
     * Thm 5 is Thm 3 over Thm 4 and at least 1 */
    nbsgd_accounting a;
    CHECK(nbsgd_iteration_accounting(times, n, m, &a) == NBSGD_OK);
    CHECK(a.x_first == timing[0] && a.x_last == timing[1]);
    CHECK(a.ratio >= 1.0 && fabs(a.ratio - a.throughput / a.throughput_sync) < 1e-12 * a.ratio);
    CHECK(a.data >= m - 1e-9 && a.data <= n * m + 1e-9);
  }
  CHECK(nbsgd_iteration_accounting(NULL, n, m, NULL) == NBSGD_E_ARG);
  /* constant delays: everybody finishes everything */
  nbsgd_delay c = {NBSGD_DELAY_CONST, 1.0, 0.0, -1, 1.0, 0.0};
  CHECK(nbsgd_sample_mask(3, 0, n, m, &c, mask, counts, NULL, NULL) == NBSGD_OK);
  for (int i = 0; i < n; ++i) CHECK(counts[i] == m);
  /* errors: null outputs, m beyond the limit, unknown kind */
  CHECK(nbsgd_sample_mask(0, 0, n, m, &d, NULL, counts, NULL, NULL) == NBSGD_E_ARG);
  CHECK(strlen(nbsgd_last_error()) > 0);
  CHECK(nbsgd_sample_mask(0, 0, n, NBSGD_MAX_MINIBATCHES + 1, &d, mask, counts, NULL, NULL) ==
        NBSGD_E_UNSUPPORTED);
  nbsgd_delay bad = d;
  bad.kind = 9;
  CHECK(nbsgd_sample_mask(0, 0, n, m, &bad, mask, counts, NULL, NULL) == NBSGD_E_ARG);
}

static void mixing(void) {
  float W[16 * 16];
  CHECK(nbsgd_w_ring(8, W) == NBSGD_OK);
  doubly_stochastic(W, 8);
  CHECK(W[0 * 8 + 7] == W[0 * 8 + 1] && W[0 * 8 + 4] == 0.0f);
  CHECK(nbsgd_w_allreduce(16, W) == NBSGD_OK);
  doubly_stochastic(W, 16);
  CHECK(nbsgd_w_ring(0, W) != NBSGD_OK && nbsgd_w_ring(4, NULL) == NBSGD_E_ARG);

  nbsgd_matcha *g = NULL;
  CHECK(nbsgd_matcha_create(0, 16, 3, &g) == NBSGD_OK && g != NULL);
  int32_t E = 0, M = 0;
  CHECK(nbsgd_matcha_matchings(g, NULL, &E, &M) == NBSGD_OK);
  CHECK(E == 24 && M >= 3 && M <= 5);
  int32_t *edges = malloc(sizeof(int32_t) * 3 * (size_t)E);
  CHECK(nbsgd_matcha_matchings(g, edges, &E, &M) == NBSGD_OK);
  int degree[16] = {0};
  for (int e = 0; e < E; ++e) {
    CHECK(edges[3 * e] < edges[3 * e + 1]);
    ++degree[edges[3 * e]];
    ++degree[edges[3 * e + 1]];
  }
  for (int v = 0; v < 16; ++v) CHECK(degree[v] == 3);
  free(edges);
  for (uint64_t step = 0; step < 10; ++step) {
    int32_t active = -1;
    CHECK(nbsgd_matcha_w(g, step, W, &active) == NBSGD_OK);
    CHECK(active >= 0 && active <= M);
    doubly_stochastic(W, 16);
  }
  double probs[8], alpha = 0.0, lam = 0.0, rho = 0.0;
  CHECK(nbsgd_matcha_optimize(g, 0.5, 500, &lam, &rho) == NBSGD_OK);
  CHECK(nbsgd_matcha_get(g, probs, &alpha) == NBSGD_OK);
  double spent = 0.0;
  for (int q = 0; q < M; ++q) {
    CHECK(probs[q] >= 0.0 && probs[q] <= 1.0);
    spent += probs[q];
  }
  CHECK(spent <= 0.5 * M + 1e-9 && alpha > 0.0 && alpha <= 1.0 / 3.0 && lam > 0.0 && rho < 1.0);
  nbsgd_matcha_destroy(g);
  CHECK(nbsgd_matcha_create(0, 5, 3, &g) == NBSGD_E_SHAPE); /* n * degree odd */
}

static void layout(void) {
  int64_t ld = -1;
  CHECK(nbsgd_row_stride(11200000, &ld) == NBSGD_OK && ld == 3 * ((int64_t)1 << 22));
  CHECK(nbsgd_row_stride(1578508, &ld) == NBSGD_OK && ld == (int64_t)1 << 21);
  CHECK(nbsgd_row_stride(1000, &ld) == NBSGD_OK && ld == 1000);
  CHECK(nbsgd_row_stride(-1, &ld) == NBSGD_E_SHAPE && nbsgd_row_stride(5, NULL) == NBSGD_E_ARG);

  nbsgd_mlp_shape s = {3072, 512, 10, 32};
  int64_t P = 0;
  size_t bytes = 0;
  CHECK(nbsgd_mlp_param_count(&s, &P) == NBSGD_OK && P == 1578508);
  CHECK(nbsgd_mlp_workspace_bytes(&s, 2048, &bytes) == NBSGD_OK && bytes > 0);
  nbsgd_mlp_shape bad = {3000, 512, 10, 32};
  CHECK(nbsgd_mlp_param_count(&bad, &P) == NBSGD_E_UNSUPPORTED);

  enum { n = 4, m = 2, b = 8, shard = 40 };
  int32_t idx[n * m * b];
  CHECK(nbsgd_minibatch_indices(1, 3, n, m, b, shard, idx) == NBSGD_OK);
  for (int i = 0; i < n; ++i) {
    int seen[shard] = {0};
    for (int k = 0; k < m * b; ++k) {
      const int32_t v = idx[i * m * b + k];
      CHECK(v >= shard * i && v < shard * (i + 1));
      if (v >= shard * i && v < shard * (i + 1)) {
        CHECK(!seen[v - shard * i]); /* a window of one permutation */
        seen[v - shard * i] = 1;
      }
    }
  }
  CHECK(nbsgd_minibatch_indices(1, 0, n, m, b, m * b - 1, idx) == NBSGD_E_SHAPE);
}

int main(void) {
  schedule();
  mixing();
  layout();
  if (failures) {
    fprintf(stderr, "%d checks failed\n", failures);
    return 1;
  }
  printf("ok\n");
  return 0;
}
