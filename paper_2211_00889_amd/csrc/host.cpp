// Host half of libnbsgd: the simulated straggler schedule, the uniform and
// ring mixing matrices, the local shuffle, argument checks and the
// thread-local error text (MATCHA is in matcha.cpp).  Built with g++ -ffp-contract=off so every fp64 operation of the
// schedule is a single IEEE operation in source order and log/pow are the
// platform libm's.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <string>
#include <vector>

#include "internal.h"

namespace nbsgd {

namespace {
thread_local std::string g_error;
}  // namespace

nbsgd_status fail(nbsgd_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_error = buf;
  return st;
}

void clear_error() { g_error.clear(); }

nbsgd_status check_nm(int32_t n, int32_t m) {
  if (n < 1 || m < 1) return fail(NBSGD_E_SHAPE, "n=%d and m=%d must be >= 1", n, m);
  if (n > NBSGD_MAX_LEARNERS)
    return fail(NBSGD_E_UNSUPPORTED, "n=%d exceeds NBSGD_MAX_LEARNERS=%d", n, NBSGD_MAX_LEARNERS);
  if (m > NBSGD_MAX_MINIBATCHES)
    return fail(NBSGD_E_UNSUPPORTED, "m=%d exceeds NBSGD_MAX_MINIBATCHES=%d", m,
                NBSGD_MAX_MINIBATCHES);
  return NBSGD_OK;
}

nbsgd_status check_w(const float* W, int32_t n) {
  if (W == nullptr) return fail(NBSGD_E_ARG, "W is null");
  for (int32_t i = 0; i < n; ++i) {
    double row = 0.0, col = 0.0;
    for (int32_t p = 0; p < n; ++p) {
      const float a = W[i * n + p];
      if (!isfinite(a) || a < 0.0f)
        return fail(NBSGD_E_W, "W[%d][%d]=%g is negative or not finite", i, p, (double)a);
      row += a;
      col += W[p * n + i];
    }
    if (fabs(row - 1.0) > 1e-5) return fail(NBSGD_E_W, "row %d of W sums to %.9g", i, row);
    if (fabs(col - 1.0) > 1e-5) return fail(NBSGD_E_W, "column %d of W sums to %.9g", i, col);
  }
  return NBSGD_OK;
}

namespace {

// ---- Philox4x64-10 (Salmon, Moraes, Dror, Shaw, SC'11) --------------------
constexpr uint64_t kMul0 = 0xD2E7470EE14C6C93ull;
constexpr uint64_t kMul1 = 0xCA5A826395121157ull;
constexpr uint64_t kBump0 = 0x9E3779B97F4A7C15ull;
constexpr uint64_t kBump1 = 0xBB67AE8584CAA73Bull;

struct Philox4x64 {
  uint64_t v[4];
};

Philox4x64 philox(uint64_t c0, uint64_t c1, uint64_t c2, uint64_t c3, uint64_t k0, uint64_t k1) {
  for (int r = 0; r < 10; ++r) {
    if (r) {
      k0 += kBump0;
      k1 += kBump1;
    }
    const unsigned __int128 a = (unsigned __int128)kMul0 * c0;
    const unsigned __int128 b = (unsigned __int128)kMul1 * c2;
    const uint64_t a_hi = (uint64_t)(a >> 64), a_lo = (uint64_t)a;
    const uint64_t b_hi = (uint64_t)(b >> 64), b_lo = (uint64_t)b;
    const uint64_t n0 = b_hi ^ c1 ^ k0, n2 = a_hi ^ c3 ^ k1;
    c0 = n0;
    c1 = b_lo;
    c2 = n2;
    c3 = a_lo;
  }
  return Philox4x64{{c0, c1, c2, c3}};
}

}  // namespace

uint64_t draw(uint64_t seed, uint64_t purpose, uint64_t c0, uint64_t c1, uint64_t c2) {
  return philox(c0, c1, c2, 0, seed, purpose).v[0];
}

double open_unit(uint64_t w) { return ((double)(w >> 12) + 0.5) * 0x1p-52; }

uint64_t below(uint64_t w, uint64_t k) { return (uint64_t)(((unsigned __int128)w * k) >> 64); }

}  // namespace nbsgd

using namespace nbsgd;

// ---------------------------------------------------------------- schedule
extern "C" nbsgd_status nbsgd_sample_mask(uint64_t seed, uint64_t step, int32_t n, int32_t m,
                                          const nbsgd_delay* d, uint8_t* mask, int32_t* counts,
                                          double* times, double* timing) {
  clear_error();
  if (nbsgd_status st = check_nm(n, m)) return st;
  if (!d || !mask || !counts) return fail(NBSGD_E_ARG, "d, mask and counts must not be null");
  if (d->kind < NBSGD_DELAY_CONST || d->kind > NBSGD_DELAY_LOMAX)
    return fail(NBSGD_E_ARG, "unknown delay kind %d", d->kind);
  if (d->kind != NBSGD_DELAY_CONST && (!(d->param > 0.0) || !isfinite(d->param)))
    return fail(NBSGD_E_ARG, "delay param %g must be finite and > 0", d->param);
  if (!(d->base >= 0.0) || !isfinite(d->base)) return fail(NBSGD_E_ARG, "delay base must be >= 0");
  if (d->slow_learner < NBSGD_SLOW_RANDOM || d->slow_learner >= n)
    return fail(NBSGD_E_ARG, "slow_learner=%d must be in [-2, n)", d->slow_learner);
  if (d->slow_learner >= 0 && (!(d->slow_factor > 0.0) || !isfinite(d->slow_factor)))
    return fail(NBSGD_E_ARG, "slow_factor %g must be finite and > 0", d->slow_factor);
  if (d->slow_learner == NBSGD_SLOW_RANDOM &&
      (!(d->slow_factor >= 1.0) || !isfinite(d->slow_factor) || !(d->slow_prob >= 0.0) ||
       !(d->slow_prob <= 1.0)))
    return fail(NBSGD_E_ARG, "random slow-down needs slow_factor >= 1 and slow_prob in [0, 1]");

  double finish[NBSGD_MAX_LEARNERS][NBSGD_MAX_MINIBATCHES] = {};
  for (int32_t i = 0; i < n; ++i) {
    double s = (i == d->slow_learner) ? d->slow_factor : 1.0;
    if (d->slow_learner == NBSGD_SLOW_RANDOM) {
      const Philox4x64 b = philox(step, (uint64_t)i, 0, 0, seed, kPurposeSlowdown);
      if (open_unit(b.v[0]) < d->slow_prob) s = 1.0 + (d->slow_factor - 1.0) * open_unit(b.v[1]);
    }
    double clock = 0.0;
    for (int32_t j = 0; j < m; ++j) {
      const double u = open_unit(draw(seed, kPurposeDelay, step, (uint64_t)i, (uint64_t)j));
      double D = 0.0;
      if (d->kind == NBSGD_DELAY_EXP)
        D = -log(u) / d->param;
      else if (d->kind == NBSGD_DELAY_LOMAX)
        D = pow(u, -1.0 / d->param) - 1.0;
      const double t = s * (d->base + D);
      clock = clock + t;
      finish[i][j] = clock;
      if (times) times[i * m + j] = t;
    }
  }
  double T = finish[0][m - 1];
  for (int32_t i = 1; i < n; ++i) T = std::min(T, finish[i][m - 1]);
  double t_sync = finish[0][m - 1], t_step = T;
  for (int32_t i = 0; i < n; ++i) {
    int32_t c = 0;
    while (c < m && finish[i][c] <= T) ++c;
    if (c == 0) c = 1;  // a learner always keeps its first mini-batch
    counts[i] = c;
    for (int32_t j = 0; j < m; ++j) mask[i * m + j] = (uint8_t)(j < c);
    t_sync = std::max(t_sync, finish[i][m - 1]);
    t_step = std::max(t_step, finish[i][c - 1]);
  }
  if (timing) {
    timing[0] = T;
    timing[1] = t_sync;
    timing[2] = t_step;
  }
  return NBSGD_OK;
}

// --------------------------------------------------- Sec. 4.3 accounting
extern "C" nbsgd_status nbsgd_iteration_accounting(const double* times, int32_t n, int32_t m,
                                                   nbsgd_accounting* out) {
  clear_error();
  if (nbsgd_status st = check_nm(n, m)) return st;
  if (!times || !out) return fail(NBSGD_E_ARG, "times and out must not be null");
  double X[NBSGD_MAX_LEARNERS];
  for (int32_t i = 0; i < n; ++i) {
    double total = 0.0;
    for (int32_t j = 0; j < m; ++j) {
      const double t = times[i * m + j];
      if (!isfinite(t) || t < 0.0)
        return fail(NBSGD_E_ARG, "times[%d][%d]=%g is negative or not finite", i, j, t);
      total = total + t;
    }
    if (!(total > 0.0)) return fail(NBSGD_E_ARG, "learner %d's batch time is not positive", i);
    X[i] = total;
  }
  // order statistics X_{1:P} <= ... <= X_{P:P}; Y summed from the fastest
  std::sort(X, X + n);
  double Y = 0.0;
  for (int32_t k = 0; k < n; ++k) Y = Y + 1.0 / X[k];
  out->x_first = X[0];
  out->x_last = X[n - 1];
  out->y = Y;
  out->throughput = (double)m * Y;
  out->throughput_sync = (double)((int64_t)n * m) / X[n - 1];
  out->data = out->throughput * X[0];
  out->ratio = (Y * X[n - 1]) / (double)n;
  return NBSGD_OK;
}

// --------------------------------------------------------- mixing matrices
extern "C" nbsgd_status nbsgd_w_allreduce(int32_t n, float* W) {
  clear_error();
  if (nbsgd_status st = check_nm(n, 1)) return st;
  if (!W) return fail(NBSGD_E_ARG, "W is null");
  const float w = (float)(1.0 / (double)n);
  for (int32_t k = 0; k < n * n; ++k) W[k] = w;
  return NBSGD_OK;
}

extern "C" nbsgd_status nbsgd_w_ring(int32_t n, float* W) {
  clear_error();
  if (nbsgd_status st = check_nm(n, 1)) return st;
  if (!W) return fail(NBSGD_E_ARG, "W is null");
  if (n <= 2) return nbsgd_w_allreduce(n, W);
  const float third = (float)(1.0 / 3.0);
  for (int32_t k = 0; k < n * n; ++k) W[k] = 0.0f;
  for (int32_t i = 0; i < n; ++i) {
    W[i * n + (i + n - 1) % n] = third;
    W[i * n + i] = third;
    W[i * n + (i + 1) % n] = third;
  }
  return NBSGD_OK;
}

extern "C" const char* nbsgd_last_error(void) { return g_error.c_str(); }

// ------------------------------------------------------------ local shuffle
namespace {

// The permutations of the last epoch asked for on this thread: every
// iteration of an epoch reads a window of the same permutations.
struct EpochPerm {
  bool valid = false;
  uint64_t seed = 0, epoch = 0;
  int32_t n = 0, shard = 0;
  std::vector<int32_t> perm;  // [n][shard]
};
thread_local EpochPerm t_perm;

const std::vector<int32_t>& epoch_permutations(uint64_t seed, uint64_t epoch, int32_t n,
                                               int32_t shard) {
  EpochPerm& e = t_perm;
  if (e.valid && e.seed == seed && e.epoch == epoch && e.n == n && e.shard == shard) return e.perm;
  e.valid = false;
  e.perm.resize((size_t)n * shard);
  for (int32_t i = 0; i < n; ++i) {
    int32_t* perm = e.perm.data() + (size_t)i * shard;
    for (int32_t t = 0; t < shard; ++t) perm[t] = t;
    for (int32_t t = shard - 1; t >= 1; --t) {
      const uint64_t r = below(draw(seed, kPurposeShuffle, epoch, (uint64_t)i, (uint64_t)t),
                               (uint64_t)t + 1);
      std::swap(perm[t], perm[r]);
    }
  }
  e.seed = seed;
  e.epoch = epoch;
  e.n = n;
  e.shard = shard;
  e.valid = true;
  return e.perm;
}

}  // namespace

extern "C" nbsgd_status nbsgd_minibatch_indices(uint64_t seed, uint64_t step, int32_t n, int32_t m,
                                                int32_t b, int32_t shard, int32_t* idx) {
  clear_error();
  if (nbsgd_status st = check_nm(n, m)) return st;
  if (!idx) return fail(NBSGD_E_ARG, "idx is null");
  if (b < 1 || shard < (int64_t)m * b)
    return fail(NBSGD_E_SHAPE, "shard=%d must hold at least m*b=%lld samples", shard,
                (long long)m * b);
  const int64_t per_epoch = shard / ((int64_t)m * b);
  const uint64_t epoch = step / (uint64_t)per_epoch;
  const int64_t window = (int64_t)(step % (uint64_t)per_epoch);
  const std::vector<int32_t>& perm = epoch_permutations(seed, epoch, n, shard);
  const int64_t base = window * m * b;
  for (int32_t i = 0; i < n; ++i)
    for (int64_t k = 0; k < (int64_t)m * b; ++k)
      idx[(int64_t)i * m * b + k] = (int32_t)((int64_t)shard * i + perm[(size_t)i * shard + base + k]);
  return NBSGD_OK;
}
