/* nbsgd_step_strided (order 0 or 1) or nbsgd_step_server (order 2, with row 0
 * of X as the server model and W unused) called from plain C on device
 * buffers from the HIP runtime: reads one step's inputs from a file, runs the
 * fused step on rows `ld` floats apart whose padding holds a sentinel, checks
 * that the padding is untouched and that misaligned and overlapping buffers
 * are rejected before any launch, and writes X and V (unpadded) to a file.
 * Used by tests/test_gpu_c_abi.py, which compares them with the oracle.
 *
 * Input, little-endian: int32 n, m, order; int64 P, ld; float lr, momentum;
 * uint8 mask[n*m]; float W[n*n], X[n*P], V[n*P], G[n*m*P].
 * Output: float X[n*P], V[n*P]. */
#include <hip/hip_runtime_api.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "nbsgd.h"

#define SENTINEL 7.0f

static int read_all(FILE *f, void *dst, size_t bytes) { return fread(dst, 1, bytes, f) == bytes; }

static int hip_ok(hipError_t e, const char *what) {
  if (e != hipSuccess) fprintf(stderr, "%s: %s\n", what, hipGetErrorString(e));
  return e == hipSuccess;
}

/* rows of `P` floats from `src` into device rows `ld` floats apart */
static int put_rows(float *dev, const float *src, int64_t rows, int64_t P, int64_t ld) {
  return hip_ok(hipMemcpy2D(dev, (size_t)ld * 4, src, (size_t)P * 4, (size_t)P * 4, (size_t)rows,
                            hipMemcpyHostToDevice),
                "hipMemcpy2D to device");
}

static int padding_intact(const float *rows, int64_t count, int64_t P, int64_t ld) {
  for (int64_t r = 0; r < count; ++r)
    for (int64_t c = P; c < ld; ++c)
      if (rows[r * ld + c] != SENTINEL) return 0;
  return 1;
}

int main(int argc, char **argv) {
  if (argc != 3) {
    fprintf(stderr, "usage: %s in.bin out.bin\n", argv[0]);
    return 2;
  }
  FILE *in = fopen(argv[1], "rb");
  if (!in) return 2;
  int32_t n, m, order;
  int64_t P, ld;
  float lr, momentum;
  if (!read_all(in, &n, 4) || !read_all(in, &m, 4) || !read_all(in, &order, 4) ||
      !read_all(in, &P, 8) || !read_all(in, &ld, 8) || !read_all(in, &lr, 4) ||
      !read_all(in, &momentum, 4))
    return 2;
  if (n < 1 || n > NBSGD_MAX_LEARNERS || m < 1 || m > NBSGD_MAX_MINIBATCHES || P < 1 || ld < P ||
      P > ((int64_t)1 << 26))
    return 2;
  const int64_t xn = (int64_t)n * P, gn = (int64_t)n * m * P;
  const int64_t xpad = (int64_t)n * ld, gpad = (int64_t)n * m * ld;
  uint8_t *mask = malloc((size_t)n * m);
  float *W = malloc(sizeof(float) * n * n);
  float *X = malloc(sizeof(float) * xn), *V = malloc(sizeof(float) * xn);
  float *G = malloc(sizeof(float) * gn);
  float *fill = malloc(sizeof(float) * gpad);
  if (!mask || !W || !X || !V || !G || !fill) return 2;
  if (!read_all(in, mask, (size_t)n * m) || !read_all(in, W, sizeof(float) * n * n) ||
      !read_all(in, X, sizeof(float) * xn) || !read_all(in, V, sizeof(float) * xn) ||
      !read_all(in, G, sizeof(float) * gn))
    return 2;
  fclose(in);
  for (int64_t k = 0; k < gpad; ++k) fill[k] = SENTINEL;

  float *dX, *dV, *dG;
  if (!hip_ok(hipMalloc((void **)&dX, sizeof(float) * xpad), "hipMalloc X") ||
      !hip_ok(hipMalloc((void **)&dV, sizeof(float) * xpad), "hipMalloc V") ||
      !hip_ok(hipMalloc((void **)&dG, sizeof(float) * gpad), "hipMalloc G"))
    return 3;
  if (!hip_ok(hipMemcpy(dX, fill, sizeof(float) * xpad, hipMemcpyHostToDevice), "fill X") ||
      !hip_ok(hipMemcpy(dV, fill, sizeof(float) * xpad, hipMemcpyHostToDevice), "fill V") ||
      !hip_ok(hipMemcpy(dG, fill, sizeof(float) * gpad, hipMemcpyHostToDevice), "fill G") ||
      !put_rows(dX, X, n, P, ld) || !put_rows(dV, V, n, P, ld) ||
      !put_rows(dG, G, (int64_t)n * m, P, ld))
    return 3;

  int failures = 0;
  const int server = order == 2;
  /* rejected before any launch: a misaligned base and X overlapping V */
  const nbsgd_status misaligned =
      server ? nbsgd_step_server(dX + 1, dV, dG, ld, mask, n, m, P, lr, momentum, NULL)
             : nbsgd_step_strided(dX + 1, dV, dG, ld, mask, W, n, m, P, lr, momentum, order, NULL);
  if (misaligned != NBSGD_E_ALIGN) {
    fprintf(stderr, "misaligned X was not rejected\n");
    ++failures;
  }
  const nbsgd_status overlap =
      server ? nbsgd_step_server(dX, dX, dG, ld, mask, n, m, P, lr, momentum, NULL)
             : nbsgd_step_strided(dX, dX, dG, ld, mask, W, n, m, P, lr, momentum, order, NULL);
  if (overlap != NBSGD_E_ARG) {
    fprintf(stderr, "X overlapping V was not rejected\n");
    ++failures;
  }
  const nbsgd_status st =
      server ? nbsgd_step_server(dX, dV, dG, ld, mask, n, m, P, lr, momentum, NULL)
             : nbsgd_step_strided(dX, dV, dG, ld, mask, W, n, m, P, lr, momentum, order, NULL);
  if (st != NBSGD_OK) {
    fprintf(stderr, "%s: status %d: %s\n", server ? "nbsgd_step_server" : "nbsgd_step_strided",
            (int)st, nbsgd_last_error());
    return 4;
  }
  if (!hip_ok(hipDeviceSynchronize(), "hipDeviceSynchronize")) return 3;
  float *outX = malloc(sizeof(float) * xpad), *outV = malloc(sizeof(float) * xpad);
  float *outG = malloc(sizeof(float) * gpad);
  if (!outX || !outV || !outG) return 2;
  if (!hip_ok(hipMemcpy(outX, dX, sizeof(float) * xpad, hipMemcpyDeviceToHost), "copy X") ||
      !hip_ok(hipMemcpy(outV, dV, sizeof(float) * xpad, hipMemcpyDeviceToHost), "copy V") ||
      !hip_ok(hipMemcpy(outG, dG, sizeof(float) * gpad, hipMemcpyDeviceToHost), "copy G"))
    return 3;
  if (!padding_intact(outX, n, P, ld) || !padding_intact(outV, n, P, ld) ||
      !padding_intact(outG, (int64_t)n * m, P, ld)) {
    fprintf(stderr, "row padding was written\n");
    ++failures;
  }
  for (int64_t k = 0; k < gn; ++k) {
    const int64_t r = k / P, c = k % P;
    if (outG[r * ld + c] != G[k]) {  /* G is read only */
      fprintf(stderr, "G changed at %lld\n", (long long)k);
      ++failures;
      break;
    }
  }
  FILE *out = fopen(argv[2], "wb");
  if (!out) return 2;
  for (int i = 0; i < n; ++i) fwrite(outX + (int64_t)i * ld, sizeof(float), (size_t)P, out);
  for (int i = 0; i < n; ++i) fwrite(outV + (int64_t)i * ld, sizeof(float), (size_t)P, out);
  fclose(out);
  hipFree(dX);
  hipFree(dV);
  hipFree(dG);
  if (failures) return 1;
  printf("ok\n");
  return 0;
}
