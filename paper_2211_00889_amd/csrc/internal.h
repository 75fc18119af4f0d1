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

}  // namespace nbsgd
