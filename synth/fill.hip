// Device side of the synthetic-input generator: fills fp32 tensors with the
// values defined in gen.py (SplitMix64 words, Irwin-Hall approximately normal
// or 24-bit uniform shaping, one correctly rounded fp32 multiply).  Holds no
// arithmetic of the optimisation method itself.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "synth.h"

namespace {

constexpr uint64_t kGamma = 0x9E3779B97F4A7C15ull;

__device__ __forceinline__ uint64_t fmix(uint64_t z) {
  z ^= z >> 30;
  z *= 0xBF58476D1CE4E5B9ull;
  z ^= z >> 27;
  z *= 0x94D049BB133111EBull;
  z ^= z >> 31;
  return z;
}

// kind 0: approximately normal, kind 1: uniform on [-a, a)
template <int KIND>
__global__ void __launch_bounds__(256) fill_kernel(float* __restrict__ dst, int64_t count,
                                                   int64_t first, uint64_t key, float scale) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count; i += stride) {
    const uint64_t e = (uint64_t)(first + i);
    const uint64_t w = fmix(key + (e + 1ull) * kGamma);
    int32_t centred;
    if (KIND == 0) {
      const uint32_t s = (uint32_t)(w & 0xFFFF) + (uint32_t)((w >> 16) & 0xFFFF) +
                         (uint32_t)((w >> 32) & 0xFFFF) + (uint32_t)(w >> 48);
      centred = (int32_t)s - 131070;
    } else {
      centred = (int32_t)(w >> 40) - 8388608;
    }
    dst[i] = (float)centred * scale;
  }
}

uint64_t fmix_host(uint64_t z) {
  z ^= z >> 30;
  z *= 0xBF58476D1CE4E5B9ull;
  z ^= z >> 27;
  z *= 0x94D049BB133111EBull;
  z ^= z >> 31;
  return z;
}

}  // namespace

extern "C" {

// Fills dst[0:count] with the generator's values for flat indices
// [first, first + count) of the tensor keyed by `key` (see gen.splitmix_key).
// Returns 0 on success, a hipError_t value otherwise.
int synth_fill(float* dst, int64_t count, int64_t first, uint64_t key, float scale, int kind,
               void* stream) {
  if (count <= 0) return 0;
  if (dst == nullptr || first < 0 || (kind != 0 && kind != 1)) return (int)hipErrorInvalidValue;
  int64_t blocks = (count + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  if (kind == 0)
    hipLaunchKernelGGL(fill_kernel<0>, dim3((unsigned)blocks), dim3(256), 0, s, dst, count, first,
                       key, scale);
  else
    hipLaunchKernelGGL(fill_kernel<1>, dim3((unsigned)blocks), dim3(256), 0, s, dst, count, first,
                       key, scale);
  return (int)hipGetLastError();
}

int synth_fill_normal(float* dst, int64_t count, int64_t first, uint64_t seed, uint64_t stream_id,
                      double std, void* stream) {
  const uint64_t key = fmix_host(fmix_host(seed + kGamma) + (stream_id + 1) * kGamma);
  // standard deviation of the centred sum of four uniform 16-bit integers
  const double unit = sqrt((65536.0 * 65536.0 - 1.0) / 3.0);
  return synth_fill(dst, count, first, key, (float)(std / unit), 0, stream);
}

}  // extern "C"
