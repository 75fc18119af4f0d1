// Internal helpers shared by the host and device translation units of libnbsgd.
#pragma once

#include <stdint.h>

#include "nbsgd.h"

namespace nbsgd {

// Records a formatted message as the calling thread's last error and returns
// `st`, so checks read `return fail(NBSGD_E_ARG, "...", ...)`.
nbsgd_status fail(nbsgd_status st, const char* fmt, ...) __attribute__((format(printf, 2, 3)));

// Resets the calling thread's error text at the start of every public call.
void clear_error();

// Checks a host mixing matrix: finite, non-negative, every row and column sum
// within 1e-5 of 1.
nbsgd_status check_w(const float* W, int32_t n);

// Checks n and m against the compiled limits.
nbsgd_status check_nm(int32_t n, int32_t m);

// Philox4x64-10 purposes (key = (seed, purpose)).
enum : uint64_t {
  kPurposeDelay = 1,
  kPurposeGraph = 2,
  kPurposeActivation = 3,
  kPurposeShuffle = 4,
  kPurposeSlowdown = 5
};

// Word 0 of Philox4x64-10 at counter (c0, c1, c2, 0) under key (seed, purpose).
uint64_t draw(uint64_t seed, uint64_t purpose, uint64_t c0, uint64_t c1, uint64_t c2);

// (0, 1): the top 52 bits of w plus one half unit, times 2^-52 (exact in fp64).
double open_unit(uint64_t w);

// [0, k): floor(w * k / 2^64).
uint64_t below(uint64_t w, uint64_t k);

}  // namespace nbsgd
