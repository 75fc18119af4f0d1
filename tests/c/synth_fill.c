/* The harness generator's C ABI (include/synth.h) from plain C.  Without a
 * GPU (argument "host"): the argument errors, returned before anything is
 * enqueued.  With a GPU (argument "device"): synth_fill_normal on a device
 * buffer, copied back and compared bit for bit with this file's own
 * transcription of the generator's definition (the SplitMix64 output
 * function and the Irwin-Hall shaping, as the header states them), at an
 * element offset, for two tensor streams.  Prints "ok" and exits 0 when
 * every check holds. */
#include <hip/hip_runtime_api.h>
#include <math.h>
#include <stdio.h>
#include <string.h>

#include "synth.h"

static uint64_t fmix(uint64_t z) {
  z ^= z >> 30;
  z *= 0xBF58476D1CE4E5B9ull;
  z ^= z >> 27;
  z *= 0x94D049BB133111EBull;
  z ^= z >> 31;
  return z;
}

static float expected(uint64_t seed, uint64_t stream_id, int64_t e, double std) {
  const uint64_t gamma = 0x9E3779B97F4A7C15ull;
  const uint64_t key = fmix(fmix(seed + gamma) + (stream_id + 1) * gamma);
  const uint64_t w = fmix(key + ((uint64_t)e + 1) * gamma);
  const int32_t s = (int32_t)((w & 0xFFFF) + ((w >> 16) & 0xFFFF) + ((w >> 32) & 0xFFFF) + (w >> 48)) -
                    131070;
  const float scale = (float)(std / sqrt((65536.0 * 65536.0 - 1.0) / 3.0));
  return (float)s * scale;
}

static int host_checks(void) {
  int bad = 0;
  float x;
  bad |= synth_fill(NULL, 4, 0, 1, 1.0f, 0, NULL) != (int)hipErrorInvalidValue;
  bad |= synth_fill(&x, 1, -1, 1, 1.0f, 0, NULL) != (int)hipErrorInvalidValue;
  bad |= synth_fill(&x, 1, 0, 1, 1.0f, 2, NULL) != (int)hipErrorInvalidValue;
  bad |= synth_fill_normal(NULL, 4, 0, 0, 1, 1.0, NULL) != (int)hipErrorInvalidValue;
  bad |= synth_fill(NULL, 0, 0, 1, 1.0f, 0, NULL) != 0; /* empty */
  bad |= synth_fill_normal(NULL, -3, 0, 0, 1, 1.0, NULL) != 0;
  return bad;
}

static int device_checks(void) {
  enum { N = 4099 };
  static float got[N];
  const int64_t first = 123456789;
  const double stds[2] = {1.0, 0.0316227766016838};
  float *d = NULL;
  if (hipMalloc((void **)&d, sizeof(float) * N) != hipSuccess) return 1;
  int bad = 0;
  for (int t = 0; t < 2; ++t) {
    const uint64_t seed = 7, stream_id = 1 + (uint64_t)t;
    if (synth_fill_normal(d, N, first, seed, stream_id, stds[t], NULL) != 0) bad = 1;
    if (hipMemcpy(got, d, sizeof got, hipMemcpyDeviceToHost) != hipSuccess) bad = 1;
    for (int64_t i = 0; i < N; ++i) {
      const float want = expected(seed, stream_id, first + i, stds[t]);
      if (memcmp(&got[i], &want, sizeof want) != 0) {
        if (!bad) fprintf(stderr, "element %lld: %.9g != %.9g\n", (long long)(first + i), got[i], want);
        bad = 1;
      }
    }
  }
  hipFree(d);
  return bad;
}

int main(int argc, char **argv) {
  const int device = argc > 1 && strcmp(argv[1], "device") == 0;
  int bad = host_checks();
  if (device) bad |= device_checks();
  if (bad) return 1;
  printf("ok\n");
  return 0;
}
