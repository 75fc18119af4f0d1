// Shape of the end-to-end MLP workload and the sizes derived from it, shared
// by the host checks (mlp_shape.cpp, plain C++) and the gradient kernels
// (mlp.hip), which receive Dims by value in their kernel arguments.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "nbsgd.h"

namespace nbsgd {

constexpr int kBatch = 32;        // mini-batch size (the MFMA K of dW1)
constexpr int kMaxHidden = 512;
constexpr int kMaxClasses = 16;   // classes fill one 16-wide MFMA tile
constexpr int kFeatBlock = 128;   // d_in features per dW1 workgroup
constexpr int kSkMaxSlices = 4;   // largest split of d_in in the forward GEMM

struct Dims {
  int32_t d_in, hidden, classes;
  int64_t P;   // padded parameters per replica
  int64_t ld;  // floats from one row of X (and of G) to the next, >= P
  int64_t off_b1, off_w2, off_b2, off_pad;
};

// Checks a shape against the supported ones (NBSGD_E_UNSUPPORTED) and fills
// *d with its offsets and padded size (ld = P).
nbsgd_status check_shape(const nbsgd_mlp_shape* s, Dims* d);

// Bytes rounded up to a multiple of 256.
inline size_t up256(size_t b) { return (b + 255) & ~(size_t)255; }

// Workspace of a call processing `rows` sample rows: the sample list, dZ1
// [rows/32][hidden][32] bf16 and kSkMaxSlices partial Z1 planes
// [rows][hidden] fp32, each 256-byte aligned.
inline size_t workspace_for(const Dims& d, int64_t rows) {
  return up256((size_t)rows * 4) + up256((size_t)rows * d.hidden * 2) +
         (size_t)kSkMaxSlices * up256((size_t)rows * d.hidden * 4);
}

}  // namespace nbsgd
