/*
 * synth.h - C ABI of libsynth, the seeded input generator of the test and
 * benchmark harness (not part of the method): fills device fp32 tensors with
 * the synthetic replicas, gradients and data of the workloads, bit for bit
 * the values the NumPy twin (synth/gen.py) returns for the same seed, tensor
 * stream and flat element index.  Holds none of the method's arithmetic.
 *
 * Definition.  fmix is the SplitMix64 output function (Steele, Lea, Flood,
 * OOPSLA 2014) and GAMMA = 0x9E3779B97F4A7C15 its increment; all arithmetic
 * is mod 2^64.  The key of tensor stream `stream_id` under `seed` is
 *   key = fmix(fmix(seed + GAMMA) + (stream_id + 1) * GAMMA),
 * and element e of the tensor draws w = fmix(key + (e + 1) * GAMMA).
 *   normal (kind 0): the four 16-bit fields of w summed, minus 2 * 65535
 *     (an Irwin-Hall sum, exact in fp32), times scale in one fp32 multiply;
 *     with scale = fp32(std / sqrt((65536^2 - 1) / 3)) the values have mean
 *     0, standard deviation std and support +-3.46 std.
 *   uniform (kind 1): (w >> 40) - 2^23, times scale = fp32(a / 2^23), on
 *     [-a, a).
 * These normals replace the Box-Muller draws the harness could use so that
 * the host and device generators agree bit for bit with no transcendental
 * function; the values never change the memory traffic of the method.
 *
 * Both calls fill dst[0 .. count) with elements first .. first + count - 1
 * of the tensor, asynchronously on `stream` (a hipStream_t as void*, NULL =
 * the null stream); dst is caller-owned device memory.  They return 0 on
 * success and a hipError_t value otherwise: hipErrorInvalidValue (1) for a
 * null dst with count > 0, first < 0 or an unknown kind, before anything is
 * enqueued; count <= 0 is a valid empty call.
 */
#ifndef SYNTH_H
#define SYNTH_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Elements of the tensor keyed by `key` (as defined above), shaped by `kind`
 * (0 normal, 1 uniform) with the fp32 `scale`. */
int synth_fill(float *dst, int64_t count, int64_t first, uint64_t key, float scale, int kind,
               void *stream);

/* Normal elements of stream `stream_id` under `seed` with standard deviation
 * `std`: synth_fill with the key and scale of the definition, computed on the
 * host.  The harness's fill of X ~ N(0, 1) and G ~ N(0, 1e-3). */
int synth_fill_normal(float *dst, int64_t count, int64_t first, uint64_t seed, uint64_t stream_id,
                      double std, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* SYNTH_H */
