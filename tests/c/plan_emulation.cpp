// CPU emulation of the fused step's use of its plan (plan.h, built by
// plan.cpp): for random, straggler-skewed, full and single-row masks up to
// n = 16, m = 64 (n * m = 1024), walks the kernel's phase 1 (each wave sums
// its segment of the finished rows, closing a partial-sum slot at every
// learner change and at the segment end) and phase 2 (each learner adds its
// slots in order) exactly as k_step does, with a random 64-bit tag per G row,
// and checks that every finished row lands in exactly its learner's slots,
// every slot is written once, the slots fit the LDS budget, and the
// per-learner constants and the CSR of W decode to the inputs.  Also built
// under AddressSanitizer and UndefinedBehaviorSanitizer by the CPU tests.
// Prints "ok" and exits 0 when every check holds.
#include <stdio.h>
#include <string.h>

#include <vector>

#include "plan.h"

using namespace nbsgd;

namespace {

int failures = 0;

#define CHECK(cond)                                                            \
  do {                                                                         \
    if (!(cond)) {                                                             \
      if (failures < 20) fprintf(stderr, "%s:%d: check failed: %s\n", __FILE__, __LINE__, #cond); \
      ++failures;                                                              \
    }                                                                          \
  } while (0)

struct Rng {
  uint64_t s;
  uint64_t next() {  // SplitMix64 (Steele, Lea, Flood)
    uint64_t z = (s += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
  }
  int below(int k) { return (int)(next() % (uint64_t)k); }
};

uint32_t byte_at(const uint32_t* w, int i) { return (w[i >> 2] >> (8 * (i & 3))) & 0xffu; }
uint32_t half_at(const uint32_t* w, int i) { return (w[i >> 1] >> (16 * (i & 1))) & 0xffffu; }

// The fused kernel's phases 1 and 2 on one column, with tags for rows.
void emulate_step(const std::vector<uint8_t>& mask, int n, int m, const StepPlan& S, int runs,
                  Rng& rng) {
  CHECK(runs >= 1 && runs <= kMaxRuns);
  CHECK((n + runs) * 64 * 16 <= 64 * 1024);  // the kernel's LDS
  const int total = S.prefix[n];
  CHECK(S.prefix[n + 1] == total);
  CHECK(S.seg[0] == 0 && S.seg[kStepWaves] == total);
  for (int w = 0; w < kStepWaves; ++w) {
    const int len = S.seg[w + 1] - S.seg[w];
    CHECK(len >= total / kStepWaves && len <= total / kStepWaves + 1);  // equal segments
  }
  std::vector<uint64_t> tag(n * m);
  for (auto& t : tag) t = rng.next();
  std::vector<uint64_t> part(runs, 0);
  std::vector<int> written(runs, 0), part_rows(runs, 0);
  for (int w = 0; w < kStepWaves; ++w) {
    const int e_end = S.seg[w + 1];
    int p = S.seg_p[w];
    int slot = S.seg_slot[w];
    CHECK(p >= 0 && p < n);
    int next = S.prefix[p + 1];
    uint64_t acc = 0;
    int rows = 0;
    bool open = false;
    for (int e = S.seg[w]; e < e_end; ++e) {
      const int row = (int)half_at(S.row, e);
      CHECK(row >= 0 && row < n * m && row / m == p && mask[row]);
      acc += tag[row];
      ++rows;
      open = true;
      if (e + 1 == next) {  // learner p's rows end here: close the run
        CHECK(slot >= 0 && slot < runs);
        if (slot >= 0 && slot < runs) {
          part[slot] = acc;
          part_rows[slot] = rows;
          ++written[slot];
        }
        acc = 0;
        rows = 0;
        open = false;
        ++slot;
        ++p;
        CHECK(p <= n);
        next = S.prefix[p + 1];
      }
    }
    if (open) {
      CHECK(slot >= 0 && slot < runs);
      if (slot >= 0 && slot < runs) {
        part[slot] = acc;
        part_rows[slot] = rows;
        ++written[slot];
      }
    }
  }
  for (int r = 0; r < runs; ++r) CHECK(written[r] == 1);
  CHECK(S.lslot[0] == 0 && S.lslot[n] == runs);
  for (int q = 0; q < n; ++q) {
    CHECK(S.lslot[q] < S.lslot[q + 1]);  // every learner has a row, so a slot
    uint64_t g = 0, want = 0;
    int got_rows = 0, c = 0;
    for (int r = S.lslot[q]; r < S.lslot[q + 1]; ++r) {
      g += part[r];
      got_rows += part_rows[r];
    }
    for (int j = 0; j < m; ++j)
      if (mask[q * m + j]) {
        want += tag[q * m + j];
        ++c;
      }
    CHECK(g == want && got_rows == c);
    CHECK(S.prefix[q + 1] - S.prefix[q] == c);
    CHECK(S.inv_c[q] == (float)(1.0 / (double)c));
    CHECK(S.eta[q] == (float)((double)0.1f * (double)c / (double)m));
  }
}

void check_learners(const std::vector<uint8_t>& mask, int n, int m) {
  Learners L;
  CHECK(learners_from_mask(mask.data(), n, m, 0.1f, &L) == NBSGD_OK);
  for (int i = 0; i < n; ++i) {
    int c = 0;
    for (int j = 0; j < m; ++j)
      if (mask[i * m + j]) {
        CHECK((int)byte_at(L.rows[i], c) == j);
        ++c;
      }
    CHECK(L.count[i] == c);
  }
}

void check_mixing(int n, Rng& rng) {
  // a random doubly stochastic W: a mixture of permutation matrices
  std::vector<float> W(n * n, 0.0f);
  const int terms = 1 + rng.below(4);
  std::vector<int> perm(n);
  for (int t = 0; t < terms; ++t) {
    for (int i = 0; i < n; ++i) perm[i] = i;
    for (int i = n - 1; i > 0; --i) std::swap(perm[i], perm[rng.below(i + 1)]);
    for (int i = 0; i < n; ++i) W[i * n + perm[i]] += 1.0f / terms;
  }
  Mixing M;
  if (mixing_from_w(W.data(), n, &M) != NBSGD_OK) return;  // rounding of 1/3 sums: skip
  std::vector<float> back(n * n, 0.0f);
  CHECK(M.start[0] == 0);
  for (int i = 0; i < n; ++i)
    for (int e = M.start[i]; e < M.start[i + 1]; ++e) back[i * n + (int)byte_at(M.col, e)] = M.w[e];
  CHECK(memcmp(back.data(), W.data(), sizeof(float) * n * n) == 0);
  bool all_equal = true;
  for (int k = 1; k < n * n; ++k) all_equal = all_equal && W[k] == W[0];
  CHECK((M.uniform != 0) == all_equal);
}

}  // namespace

int main() {
  Rng rng{12345};
  int cases = 0;
  for (int trial = 0; trial < 20000; ++trial) {
    const int n = 1 + rng.below(16), m = 1 + rng.below(64);
    std::vector<uint8_t> mask(n * m, 0);
    switch (trial % 5) {
      case 0:  // random, any pattern
        for (auto& b : mask) b = (uint8_t)(rng.below(3) != 0);
        break;
      case 1:  // prefix masks of random counts
        for (int i = 0; i < n; ++i) {
          const int c = 1 + rng.below(m);
          for (int j = 0; j < c; ++j) mask[i * m + j] = 1;
        }
        break;
      case 2:  // straggler-skewed: one learner finished all, the rest one or two
        for (int i = 0; i < n; ++i) {
          const int c = (i == trial % n) ? m : 1 + rng.below(2 < m ? 2 : m);
          for (int j = 0; j < c; ++j) mask[i * m + j] = 1;
        }
        break;
      case 3:  // sparse: one random mini-batch per learner
        for (int i = 0; i < n; ++i) mask[i * m + rng.below(m)] = 1;
        break;
      default:  // full
        for (auto& b : mask) b = 1;
        break;
    }
    for (int i = 0; i < n; ++i) {  // every learner keeps at least one
      bool any = false;
      for (int j = 0; j < m; ++j) any = any || mask[i * m + j];
      if (!any) mask[i * m + rng.below(m)] = 1;
    }
    StepPlan S;
    int runs = -1;
    CHECK(plan_from_mask(mask.data(), n, m, 0.1f, &S, &runs) == NBSGD_OK);
    emulate_step(mask, n, m, S, runs, rng);
    check_learners(mask, n, m);
    check_mixing(n, rng);
    ++cases;
  }
  // the largest plan: 16 learners, 64 mini-batches, every row finished
  {
    std::vector<uint8_t> mask(16 * 64, 1);
    StepPlan S;
    int runs = -1;
    CHECK(plan_from_mask(mask.data(), 16, 64, 0.1f, &S, &runs) == NBSGD_OK);
    emulate_step(mask, 16, 64, S, runs, rng);
    ++cases;
  }
  // the emulation is not vacuous: plans with a planted mistake fail it
  {
    std::vector<uint8_t> mask(6 * 10, 0);
    for (int i = 0; i < 6; ++i)
      for (int j = 0; j <= i; ++j) mask[i * 10 + j] = 1;  // counts 1..6, 21 rows
    for (int mistake = 0; mistake < 4; ++mistake) {
      StepPlan S;
      int runs = -1;
      CHECK(plan_from_mask(mask.data(), 6, 10, 0.1f, &S, &runs) == NBSGD_OK);
      if (mistake == 0) S.lslot[3] += 1;                         // a slot given to the wrong learner
      if (mistake == 1) S.seg[4] += 1;                           // overlapping segments
      if (mistake == 2) S.prefix[2] -= 1;                        // a run closed one row early
      if (mistake == 3) S.row[5] ^= 1u;                          // a wrong G row
      const int before = failures;
      emulate_step(mask, 6, 10, S, runs, rng);
      const bool caught = failures > before;
      failures = before;
      CHECK(caught);
    }
  }
  // a learner with nothing finished is refused
  {
    std::vector<uint8_t> mask(4 * 4, 1);
    for (int j = 0; j < 4; ++j) mask[2 * 4 + j] = 0;
    StepPlan S;
    int runs = -1;
    CHECK(plan_from_mask(mask.data(), 4, 4, 0.1f, &S, &runs) == NBSGD_E_MASK);
    Learners L;
    CHECK(learners_from_mask(mask.data(), 4, 4, 0.1f, &L) == NBSGD_E_MASK);
  }
  if (failures) {
    fprintf(stderr, "%d checks failed over %d plans\n", failures, cases);
    return 1;
  }
  printf("ok\n");
  return 0;
}
