// Per-step constants of the step kernels, built on the host (plan.cpp, plain
// C++) and passed by value in the kernel arguments (step.hip).  Plain structs
// of 32-bit fields, so g++ and hipcc lay them out identically; sub-word lists
// are packed into 32-bit words (the kernels read kernel arguments only as
// aligned 32-bit words).
#pragma once

#include <stdint.h>

#include "nbsgd.h"

namespace nbsgd {

constexpr int kMaxN = NBSGD_MAX_LEARNERS;
constexpr int kMaxM = NBSGD_MAX_MINIBATCHES;

// Waves per workgroup of the fused step; each takes one contiguous segment of
// the tile's finished rows.
constexpr int kStepWaves = 8;
constexpr int kMaxRows = kMaxN * kMaxM;           // finished rows of one step
constexpr int kMaxRuns = kMaxN + kStepWaves - 1;  // partial-sum slots of one tile

// Per-learner constants of the unfused stages.
struct Learners {
  float eta[kMaxN];      // lr * c_i / m
  float inv_c[kMaxN];    // 1 / c_i
  int32_t count[kMaxN];  // c_i
  // indices of the finished mini-batches in order, 8 bits each: index r of
  // learner p in byte r % 4 of rows[p][r / 4]
  uint32_t rows[kMaxN][kMaxM / 4];
};

// Mixing matrix as CSR over its nonzero entries, or the uniform flag.
struct Mixing {
  int32_t uniform;  // all entries equal: out = (sum_p z_p) * w_all
  float w_all;
  int32_t start[kMaxN + 1];         // entries of row i: [start[i], start[i+1])
  uint32_t col[kMaxN * kMaxN / 4];  // column of entry e in byte e % 4 of word e / 4
  float w[kMaxN * kMaxN];
};

// Plan of the fused step.  Entries are the finished (learner, mini-batch)
// pairs in learner-major order; wave w sums entries [seg[w], seg[w+1]).  A
// run is a maximal stretch of one learner's entries inside one wave's
// segment; runs are numbered in entry order and each owns one LDS slot, and
// learner p's runs are the slots [lslot[p], lslot[p+1]).
struct StepPlan {
  float eta[kMaxN];                   // lr * c_i / m
  float inv_c[kMaxN];                 // 1 / c_i
  int32_t prefix[kMaxN + 2];          // first entry of each learner; [n] = [n+1] = total
  int32_t seg[kStepWaves + 1];        // first entry of each wave's segment
  int32_t seg_p[kStepWaves];          // learner of a segment's first entry
  int32_t seg_slot[kStepWaves];       // slot of a segment's first run
  int32_t lslot[kMaxN + 1];           // slots of learner p: [lslot[p], lslot[p+1])
  uint32_t row[(kMaxRows + 16) / 2];  // G row (p * m + j) of entry e in half e % 2 of word e / 2
};

// Per-learner constants from a host mask [n*m] (any pattern); every learner
// needs at least one finished mini-batch (NBSGD_E_MASK).  eta_i and 1/c_i are
// formed in fp64 and rounded once.
nbsgd_status learners_from_mask(const uint8_t* mask, int32_t n, int32_t m, float lr, Learners* L);

// CSR of a checked host W [n*n] (check_w), and whether all entries are equal.
nbsgd_status mixing_from_w(const float* W, int32_t n, Mixing* out);

// The fused step's plan for a host mask [n*m]; *runs receives the number of
// LDS slots (at most kMaxRuns).
nbsgd_status plan_from_mask(const uint8_t* mask, int32_t n, int32_t m, float lr, StepPlan* S,
                            int* runs);

}  // namespace nbsgd
