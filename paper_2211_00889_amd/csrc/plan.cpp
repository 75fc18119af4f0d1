// Host planning of the step kernels (plain C++, no HIP): per-learner constants
// from the finished mask, the CSR form of W, the fused step's per-wave
// segments and partial-sum slots, and the row stride the step workloads
// allocate with.  Built with g++, so the CPU tests emulate and sanitize
// exactly the code that plans every launch.
#include "plan.h"

#include <string.h>

#include "internal.h"

namespace nbsgd {

namespace {

void set_byte(uint32_t* words, int i, uint32_t v) { words[i >> 2] |= (v & 0xffu) << (8 * (i & 3)); }
void set_half(uint32_t* words, int i, uint32_t v) {
  words[i >> 1] |= (v & 0xffffu) << (16 * (i & 1));
}

}  // namespace

nbsgd_status learners_from_mask(const uint8_t* mask, int32_t n, int32_t m, float lr, Learners* L) {
  if (!mask) return fail(NBSGD_E_ARG, "mask is null");
  memset(L, 0, sizeof *L);
  for (int32_t i = 0; i < n; ++i) {
    int32_t c = 0;
    for (int32_t j = 0; j < m; ++j)
      if (mask[i * m + j]) set_byte(L->rows[i], c++, (uint32_t)j);
    if (c == 0) return fail(NBSGD_E_MASK, "learner %d finished no mini-batch", i);
    L->count[i] = c;
    L->inv_c[i] = (float)(1.0 / (double)c);
    L->eta[i] = (float)((double)lr * (double)c / (double)m);
  }
  return NBSGD_OK;
}

nbsgd_status mixing_from_w(const float* Wh, int32_t n, Mixing* W) {
  if (nbsgd_status st = check_w(Wh, n)) return st;
  memset(W, 0, sizeof *W);
  W->uniform = 1;
  for (int32_t k = 1; k < n * n; ++k)
    if (Wh[k] != Wh[0]) W->uniform = 0;
  W->w_all = Wh[0];
  int32_t e = 0;
  for (int32_t i = 0; i < n; ++i) {
    W->start[i] = e;
    for (int32_t p = 0; p < n; ++p)
      if (Wh[i * n + p] != 0.0f) {
        set_byte(W->col, e, (uint32_t)p);
        W->w[e] = Wh[i * n + p];
        ++e;
      }
  }
  W->start[n] = e;
  return NBSGD_OK;
}

nbsgd_status plan_from_mask(const uint8_t* mask, int32_t n, int32_t m, float lr, StepPlan* S,
                            int* runs) {
  if (!mask) return fail(NBSGD_E_ARG, "mask is null");
  memset(S, 0, sizeof *S);
  int32_t e = 0;
  int learner_of[kMaxRows];
  for (int32_t i = 0; i < n; ++i) {
    S->prefix[i] = e;
    for (int32_t j = 0; j < m; ++j)
      if (mask[i * m + j]) {
        learner_of[e] = i;
        set_half(S->row, e++, (uint32_t)(i * m + j));
      }
    const int32_t c = e - S->prefix[i];
    if (c == 0) return fail(NBSGD_E_MASK, "learner %d finished no mini-batch", i);
    S->inv_c[i] = (float)(1.0 / (double)c);
    S->eta[i] = (float)((double)lr * (double)c / (double)m);
  }
  S->prefix[n] = S->prefix[n + 1] = e;
  // equal contiguous segments of the entries, one per wave; a new run (slot)
  // starts at every segment start and at every learner change inside one
  int slot = 0, last_learner = -1;
  for (int w = 0; w <= kStepWaves; ++w) S->seg[w] = (int32_t)((int64_t)w * e / kStepWaves);
  for (int w = 0; w < kStepWaves; ++w) {
    S->seg_slot[w] = slot;
    if (S->seg[w] == S->seg[w + 1]) continue;
    S->seg_p[w] = learner_of[S->seg[w]];
    for (int32_t k = S->seg[w]; k < S->seg[w + 1]; ++k) {
      const bool starts_run = k == S->seg[w] || learner_of[k] != learner_of[k - 1];
      if (!starts_run) continue;
      while (last_learner < learner_of[k]) S->lslot[++last_learner] = slot;
      ++slot;
    }
  }
  while (last_learner < n) S->lslot[++last_learner] = slot;
  *runs = slot;
  return NBSGD_OK;
}

}  // namespace nbsgd

using namespace nbsgd;

// Row strides of nbsgd_row_stride: rows longer than 2^22 floats (16 MiB)
// start on 16 MiB boundaries; rows of 2^20 floats or fewer are not padded.
namespace {
constexpr int64_t kRowAlign = int64_t(1) << 22;
constexpr int64_t kSmallRow = int64_t(1) << 20;
}  // namespace

extern "C" nbsgd_status nbsgd_row_stride(int64_t P, int64_t* ld) {
  clear_error();
  if (!ld) return fail(NBSGD_E_ARG, "ld is null");
  if (P < 0) return fail(NBSGD_E_SHAPE, "P=%lld is negative", (long long)P);
  if (P <= kSmallRow) {
    *ld = P;
    return NBSGD_OK;
  }
  if (P <= kRowAlign) {  // the next power of two, 2^21 or 2^22
    int64_t p2 = kSmallRow;
    while (p2 < P) p2 <<= 1;
    *ld = p2;
    return NBSGD_OK;
  }
  int64_t k = (P + kRowAlign - 1) / kRowAlign;  // rows of k * 2^22 floats, k >= 2
  if ((k & (k - 1)) == 0) ++k;  // a power-of-two stride aliases
  *ld = k * kRowAlign;
  return NBSGD_OK;
}
