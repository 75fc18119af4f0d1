// Device half of libnbsgd for gfx950: the fused Non-blocking step and its three
// unfused stages (accumulate, mix, update), with their argument checks.
//
// Data layout (all fp32, row-major, caller-owned HBM):
//   X, V  [n][ld]     replicas and momentum buffers, learner-major
//   G     [n][m][ld]  per-mini-batch gradients
// with rows ld >= P floats apart: the first P floats of a row are the
// parameters and the rest is never touched (ld = P except in the strided
// fused step).
// Every kernel works on column tiles: the mix couples learners, never
// columns, so a workgroup that holds all n rows of its columns can update X in
// place.  Rows are streamed as VEC-wide vectors (VEC = 4 when P % 4 == 0, else
// 2 or 1), so each wave moves 64 * VEC * 4 contiguous bytes per row per load.
//
// Fused step, one workgroup = 8 waves x 64 lanes, one VEC-vector column per
// lane, all n learners; workgroups take the column tiles from the last to the
// first (the order never changes a result: columns are independent):
//   phase 1: the finished gradient rows of the tile (sum_i c_i of them, in
//            learner-major order) are split into 8 equal contiguous segments,
//            one per wave, so a straggler-skewed mask (one learner with all m
//            rows, another with one) still gives every wave the same number
//            of loads.  A wave sums each learner's rows within its segment and
//            writes the partial sum to an LDS slot; wave w also loads X and V
//            of learners w and w + 8 into registers.
//   phase 2: wave w adds the slots of its learners in slot order (a fixed
//            order, so results are bitwise reproducible), forms the momentum
//            (stored at once) and the value to be mixed, z_p = x_p
//            (mix-then-step) or x_p - eta_p v_p (step-then-mix), into LDS;
//   phase 3: wave w forms row i = w, w + 8 of the mix from LDS (CSR of the
//            nonzero W entries, or one sum scaled by 1/n for uniform W) and
//            writes X[i].
// HBM traffic per step is the finished rows of G once, X and V read once and
// written once: 4 * P * (sum_i c_i + 4 n) bytes.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>
#include <string.h>

#include <algorithm>

#include "internal.h"
#include "plan.h"

using namespace nbsgd;

namespace {

constexpr int kWave = 64;
constexpr int kWaves = 4;
constexpr int kBlock = kWave * kWaves;
// fused step kernel shape (kStepWaves, kMaxRuns: plan.h)
constexpr int kStepBlock = kWave * kStepWaves;
constexpr int kStepSlots = (kMaxN + kStepWaves - 1) / kStepWaves;
// the fused step's LDS: n rows of values to mix and one row per run, 64 lanes
// of float4 each; within the 64 KiB a workgroup may allocate
static_assert((kMaxN + kMaxRuns) * kWave * 4 * sizeof(float) <= 64 * 1024,
              "fused step LDS exceeds 64 KiB");

template <int VEC>
struct Vec;
template <>
struct Vec<4> {
  typedef float type __attribute__((ext_vector_type(4)));
};
template <>
struct Vec<2> {
  typedef float type __attribute__((ext_vector_type(2)));
};
template <>
struct Vec<1> {
  typedef float type;
};

// Kernel arguments are only ever read as naturally aligned 32-bit words:
// sub-word arrays are packed into uint32_t and unpacked with shifts.  (A
// dynamically indexed uint8_t array next to 32-bit fields let the compiler
// form a scalar-load base address that was not 4-byte aligned; the scalar
// memory unit ignores the low two address bits, so neighbouring fields were
// read one element early.)
__device__ __forceinline__ uint32_t byte_of(const uint32_t* words, int i) {
  return (words[i >> 2] >> (8 * (i & 3))) & 0xffu;
}
__device__ __forceinline__ uint32_t half_of(const uint32_t* words, int i) {
  return (words[i >> 1] >> (16 * (i & 1))) & 0xffffu;
}

__device__ __forceinline__ int row_of(const Learners& L, int p, int r) {
  return (int)byte_of(L.rows[p], r);
}

template <typename T>
__device__ __forceinline__ T ld_stream(const T* p) {
  return __builtin_nontemporal_load(p);
}
template <typename T>
__device__ __forceinline__ void st_stream(T* p, T v) {
  __builtin_nontemporal_store(v, p);
}

// Number of finished-row loads a thread keeps in flight before summing them.
constexpr int kChunk = 16;

// Sum of the finished rows of learner p at vector column v.  Rows are loaded
// kChunk at a time (the tail chunk predicated on the uniform count) so each
// wave has kChunk independent 64 x VEC x 4-byte loads in flight.
template <int VEC>
__device__ __forceinline__ typename Vec<VEC>::type finished_sum(const typename Vec<VEC>::type* G,
                                                                const Learners& L, int p, int m,
                                                                int64_t pv, int64_t v) {
  using vf = typename Vec<VEC>::type;
  const vf* g = G + (int64_t)p * m * pv + v;
  const int c = L.count[p];
  vf acc = (vf)(0.0f);
  for (int r = 0; r < c; r += kChunk) {
    vf a[kChunk];
#pragma unroll
    for (int k = 0; k < kChunk; ++k)
      a[k] = (r + k < c) ? ld_stream(g + (int64_t)row_of(L, p, r + k) * pv) : (vf)(0.0f);
#pragma unroll
    for (int w = 1; w < kChunk; w *= 2)
#pragma unroll
      for (int k = 0; k < kChunk; k += 2 * w) a[k] += a[k + w];
    acc += a[0];
  }
  return acc;
}

// Row i of the mix at LDS column t.
template <int VEC>
__device__ __forceinline__ typename Vec<VEC>::type mix_row(const typename Vec<VEC>::type* zs,
                                                           int ncols, const Mixing& W, int i,
                                                           int t) {
  using vf = typename Vec<VEC>::type;
  vf acc = (vf)(0.0f);
  for (int e = W.start[i]; e < W.start[i + 1]; ++e)
    acc += W.w[e] * zs[(int)byte_of(W.col, e) * ncols + t];
  return acc;
}

template <int VEC>
__device__ __forceinline__ typename Vec<VEC>::type mix_all(const typename Vec<VEC>::type* zs,
                                                           int ncols, int n, int t) {
  using vf = typename Vec<VEC>::type;
  vf acc = (vf)(0.0f);
  for (int k = 0; k < n; ++k) acc += zs[k * ncols + t];
  return acc;
}

// The parameter-server form of the step (Alg. 3): X is the one server row,
// and the new server model is x - (1/n) sum_p eta_p v_p.
constexpr int kServer = 2;

template <int VEC, int ORDER>
__global__ void __launch_bounds__(kStepBlock)
    k_step(float* __restrict__ Xf, float* __restrict__ Vf, const float* __restrict__ Gf,
           int64_t pv, int64_t ldv, int n, float mu, StepPlan S, Mixing W) {
  using vf = typename Vec<VEC>::type;
  extern __shared__ char smem[];
  vf* zs = reinterpret_cast<vf*>(smem);        // [n][64]: values to be mixed
  vf* part = zs + n * kWave;                   // [runs][64]: partial row sums
  vf* X = reinterpret_cast<vf*>(Xf);
  vf* V = reinterpret_cast<vf*>(Vf);
  const vf* G = reinterpret_cast<const vf*>(Gf);

  const int lane = threadIdx.x & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  // tiles in decreasing column order: gradient rows written just before in
  // increasing column order (the MLP gradient kernels) are read newest first,
  // while the memory-side cache may still hold them
  const int64_t v = (int64_t)(gridDim.x - 1 - blockIdx.x) * kWave + lane;
  const bool live = v < pv;

  // phase 1: own learners' X and V, and this wave's share of the G rows
  vf xo[kStepSlots], vo[kStepSlots];
#pragma unroll
  for (int s = 0; s < kStepSlots; ++s) {
    const int p = wave + kStepWaves * s;
    xo[s] = (vf)(0.0f);
    vo[s] = (vf)(0.0f);
    if (p < n && live) {
      if (ORDER != kServer || p == 0) xo[s] = ld_stream(X + (int64_t)p * ldv + v);
      vo[s] = ld_stream(V + (int64_t)p * ldv + v);
    }
  }
  const int e_end = S.seg[wave + 1];
  int p = S.seg_p[wave];
  int slot = S.seg_slot[wave];
  int next = S.prefix[p + 1];  // entry where learner p's rows end
  vf acc = (vf)(0.0f);
  bool open = false;
  for (int e = S.seg[wave]; e < e_end; e += kChunk) {
    vf a[kChunk];
#pragma unroll
    for (int k = 0; k < kChunk; ++k) {
      const int64_t row = (e + k < e_end) ? (int64_t)half_of(S.row, e + k) : 0;  // uniform
      a[k] = (e + k < e_end && live) ? ld_stream(G + row * ldv + v) : (vf)(0.0f);
    }
#pragma unroll
    for (int k = 0; k < kChunk; ++k) {
      if (e + k < e_end) {
        acc += a[k];
        open = true;
        if (e + k + 1 == next) {  // learner p's rows end here: close the run
          part[slot * kWave + lane] = acc;
          acc = (vf)(0.0f);
          open = false;
          ++slot;
          ++p;
          next = S.prefix[p + 1];
        }
      }
    }
  }
  if (open) part[slot * kWave + lane] = acc;
  __syncthreads();

  // phase 2: combine partial sums in slot order, momentum, value to be mixed
  vf keep[kStepSlots];  // eta_i * v_i for mix-then-step
#pragma unroll
  for (int s = 0; s < kStepSlots; ++s) {
    const int q = wave + kStepWaves * s;
    if (q < n) {
      vf g = (vf)(0.0f);
      for (int r = S.lslot[q]; r < S.lslot[q + 1]; ++r) g += part[r * kWave + lane];
      const vf vn = mu * vo[s] + g * S.inv_c[q];
      if (live) st_stream(V + (int64_t)q * ldv + v, vn);
      if (ORDER == NBSGD_MIX_THEN_STEP) {
        zs[q * kWave + lane] = xo[s];
        keep[s] = S.eta[q] * vn;
      } else if (ORDER == NBSGD_STEP_THEN_MIX) {
        zs[q * kWave + lane] = xo[s] - S.eta[q] * vn;
      } else {  // kServer: the learner's contribution eta_q v_q
        zs[q * kWave + lane] = S.eta[q] * vn;
      }
    }
  }
  __syncthreads();

  // phase 3: mix and write the new replicas (the server row: wave 0 only)
  if (ORDER == kServer) {
    if (wave == 0 && live) st_stream(X + v, xo[0] - mix_all<VEC>(zs, kWave, n, lane) * W.w_all);
    return;
  }
  vf total = (vf)(0.0f);
  if (W.uniform) total = mix_all<VEC>(zs, kWave, n, lane) * W.w_all;
#pragma unroll
  for (int s = 0; s < kStepSlots; ++s) {
    const int i = wave + kStepWaves * s;
    if (i < n && live) {
      vf x = W.uniform ? total : mix_row<VEC>(zs, kWave, W, i, lane);
      if (ORDER == NBSGD_MIX_THEN_STEP) x -= keep[s];
      st_stream(X + (int64_t)i * ldv + v, x);
    }
  }
}

// Gbar[p] = (1/c_p) * sum of the finished rows of G[p]; blockIdx.y = learner.
template <int VEC>
__global__ void __launch_bounds__(kBlock)
    k_accumulate(const float* __restrict__ Gf, float* __restrict__ Of, int64_t pv, int m,
                 Learners L) {
  using vf = typename Vec<VEC>::type;
  const int p = blockIdx.y;
  const int64_t v = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  if (v >= pv) return;
  const vf g = finished_sum<VEC>(reinterpret_cast<const vf*>(Gf), L, p, m, pv, v);
  st_stream(reinterpret_cast<vf*>(Of) + (int64_t)p * pv + v, g * L.inv_c[p]);
}

// V[p] = mu V[p] + Gbar[p]; X[p] -= eta_p V[p]; blockIdx.y = learner.
template <int VEC>
__global__ void __launch_bounds__(kBlock)
    k_update(float* __restrict__ Xf, float* __restrict__ Vf, const float* __restrict__ Bf,
             int64_t pv, float mu, Learners L) {
  using vf = typename Vec<VEC>::type;
  const int p = blockIdx.y;
  const int64_t v = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  if (v >= pv) return;
  const int64_t off = (int64_t)p * pv + v;
  vf* X = reinterpret_cast<vf*>(Xf);
  vf* V = reinterpret_cast<vf*>(Vf);
  const vf vn = mu * ld_stream(V + off) + ld_stream(reinterpret_cast<const vf*>(Bf) + off);
  st_stream(V + off, vn);
  st_stream(X + off, ld_stream(X + off) - L.eta[p] * vn);
}

// Y = W X through an LDS tile of all n rows; Y may equal X.
template <int VEC>
__global__ void __launch_bounds__(kBlock)
    k_mix(const float* Xf, float* Yf, int64_t pv, int n, Mixing W) {
  using vf = typename Vec<VEC>::type;
  extern __shared__ char smem[];
  vf* zs = reinterpret_cast<vf*>(smem);
  constexpr int ncols = kWave;
  const vf* X = reinterpret_cast<const vf*>(Xf);
  vf* Y = reinterpret_cast<vf*>(Yf);
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int64_t v = (int64_t)blockIdx.x * ncols + lane;
  for (int p = wave; p < n; p += kWaves)
    if (v < pv) zs[p * ncols + lane] = ld_stream(X + (int64_t)p * pv + v);
  __syncthreads();
  if (v >= pv) return;
  vf total = (vf)(0.0f);
  if (W.uniform) total = mix_all<VEC>(zs, ncols, n, lane) * W.w_all;
  for (int i = wave; i < n; i += kWaves) {
    const vf y = W.uniform ? total : mix_row<VEC>(zs, ncols, W, i, lane);
    st_stream(Y + (int64_t)i * pv + v, y);
  }
}

// ------------------------------------------------------------------ host

int vec_width(int64_t P) { return (P % 4 == 0) ? 4 : (P % 2 == 0) ? 2 : 1; }

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

bool overlap(const void* a, int64_t a_bytes, const void* b, int64_t b_bytes) {
  const uintptr_t a0 = (uintptr_t)a, b0 = (uintptr_t)b;
  return a0 < b0 + (uintptr_t)b_bytes && b0 < a0 + (uintptr_t)a_bytes;
}

nbsgd_status check_launch(const char* what) {
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(NBSGD_E_HIP, "%s launch failed: %s", what, hipGetErrorString(e));
  return NBSGD_OK;
}

nbsgd_status check_rows(const void* p, const char* name) {
  if (!p) return fail(NBSGD_E_ARG, "%s is null", name);
  if (!aligned16(p)) return fail(NBSGD_E_ALIGN, "%s is not 16-byte aligned", name);
  return NBSGD_OK;
}

static_assert(sizeof(StepPlan) + sizeof(Mixing) + 64 <= 4096, "kernel arguments exceed 4 KiB");

template <int VEC, int ORDER>
void launch_step(float* X, float* V, const float* G, int64_t pv, int64_t ldv, int n, float mu,
                 const StepPlan& S, int runs, const Mixing& W, hipStream_t s) {
  const int64_t blocks = (pv + kWave - 1) / kWave;
  const size_t lds = (size_t)(n + runs) * kWave * VEC * sizeof(float);
  hipLaunchKernelGGL((k_step<VEC, ORDER>), dim3((unsigned)blocks), dim3(kStepBlock), lds, s, X,
                     V, G, pv, ldv, n, mu, S, W);
}

// The fused step on rows `ld` floats apart (ld >= P).
nbsgd_status step_impl(float* X, float* V, const float* G, int64_t ld, const uint8_t* mask,
                       const float* Wh, int32_t n, int32_t m, int64_t P, float lr, float momentum,
                       int32_t order, void* stream) {
  if (nbsgd_status st = check_nm(n, m)) return st;
  if (P < 0) return fail(NBSGD_E_SHAPE, "P=%lld is negative", (long long)P);
  if (ld < P) return fail(NBSGD_E_SHAPE, "row stride %lld is below P=%lld", (long long)ld, (long long)P);
  if (order != NBSGD_MIX_THEN_STEP && order != NBSGD_STEP_THEN_MIX)
    return fail(NBSGD_E_ARG, "unknown order %d", order);
  StepPlan S;
  int runs = 0;
  if (nbsgd_status st = plan_from_mask(mask, n, m, lr, &S, &runs)) return st;
  Mixing W;
  if (nbsgd_status st = mixing_from_w(Wh, n, &W)) return st;
  if (P == 0) return NBSGD_OK;
  if (nbsgd_status st = check_rows(X, "X")) return st;
  if (nbsgd_status st = check_rows(V, "V")) return st;
  if (nbsgd_status st = check_rows(G, "G")) return st;
  // extents: the last row needs only P floats
  const int64_t xb = ((int64_t)(n - 1) * ld + P) * 4, gb = ((int64_t)n * m - 1) * ld * 4 + P * 4;
  if (overlap(X, xb, V, xb)) return fail(NBSGD_E_ARG, "X and V overlap");
  if (overlap(G, gb, X, xb) || overlap(G, gb, V, xb))
    return fail(NBSGD_E_ARG, "G overlaps X or V");
  const int vec = std::min(vec_width(P), vec_width(ld));  // divides both P and ld
  const int64_t pv = P / vec, ldv = ld / vec;
  if ((pv + kWave - 1) / kWave > 0x7fffffff)
    return fail(NBSGD_E_UNSUPPORTED, "P=%lld needs too many workgroups", (long long)P);
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  if (order == NBSGD_MIX_THEN_STEP) {
    if (vec == 4) launch_step<4, NBSGD_MIX_THEN_STEP>(X, V, G, pv, ldv, n, momentum, S, runs, W, s);
    else if (vec == 2) launch_step<2, NBSGD_MIX_THEN_STEP>(X, V, G, pv, ldv, n, momentum, S, runs, W, s);
    else launch_step<1, NBSGD_MIX_THEN_STEP>(X, V, G, pv, ldv, n, momentum, S, runs, W, s);
  } else {
    if (vec == 4) launch_step<4, NBSGD_STEP_THEN_MIX>(X, V, G, pv, ldv, n, momentum, S, runs, W, s);
    else if (vec == 2) launch_step<2, NBSGD_STEP_THEN_MIX>(X, V, G, pv, ldv, n, momentum, S, runs, W, s);
    else launch_step<1, NBSGD_STEP_THEN_MIX>(X, V, G, pv, ldv, n, momentum, S, runs, W, s);
  }
  return check_launch("nbsgd_step");
}

}  // namespace

extern "C" nbsgd_status nbsgd_step(float* X, float* V, const float* G, const uint8_t* mask,
                                   const float* Wh, int32_t n, int32_t m, int64_t P, float lr,
                                   float momentum, int32_t order, void* stream) {
  clear_error();
  return step_impl(X, V, G, P, mask, Wh, n, m, P, lr, momentum, order, stream);
}

extern "C" nbsgd_status nbsgd_step_strided(float* X, float* V, const float* G, int64_t ld,
                                           const uint8_t* mask, const float* Wh, int32_t n,
                                           int32_t m, int64_t P, float lr, float momentum,
                                           int32_t order, void* stream) {
  clear_error();
  return step_impl(X, V, G, ld, mask, Wh, n, m, P, lr, momentum, order, stream);
}

extern "C" nbsgd_status nbsgd_step_server(float* x, float* V, const float* G, int64_t ld,
                                          const uint8_t* mask, int32_t n, int32_t m, int64_t P,
                                          float lr, float momentum, void* stream) {
  clear_error();
  if (nbsgd_status st = check_nm(n, m)) return st;
  if (P < 0) return fail(NBSGD_E_SHAPE, "P=%lld is negative", (long long)P);
  if (ld < P) return fail(NBSGD_E_SHAPE, "row stride %lld is below P=%lld", (long long)ld, (long long)P);
  StepPlan S;
  int runs = 0;
  if (nbsgd_status st = plan_from_mask(mask, n, m, lr, &S, &runs)) return st;
  Mixing W;  // the average over the n learners: 1/n, rounded once
  memset(&W, 0, sizeof W);
  W.uniform = 1;
  W.w_all = (float)(1.0 / (double)n);
  if (P == 0) return NBSGD_OK;
  if (nbsgd_status st = check_rows(x, "x")) return st;
  if (nbsgd_status st = check_rows(V, "V")) return st;
  if (nbsgd_status st = check_rows(G, "G")) return st;
  const int64_t vb = ((int64_t)(n - 1) * ld + P) * 4, gb = ((int64_t)n * m - 1) * ld * 4 + P * 4;
  if (overlap(x, P * 4, V, vb)) return fail(NBSGD_E_ARG, "x and V overlap");
  if (overlap(G, gb, x, P * 4) || overlap(G, gb, V, vb)) return fail(NBSGD_E_ARG, "G overlaps x or V");
  const int vec = std::min(vec_width(P), vec_width(ld));
  const int64_t pv = P / vec, ldv = ld / vec;
  if ((pv + kWave - 1) / kWave > 0x7fffffff)
    return fail(NBSGD_E_UNSUPPORTED, "P=%lld needs too many workgroups", (long long)P);
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  // x is a single row: the kernel reads and writes row 0 only
  if (vec == 4) launch_step<4, kServer>(x, V, G, pv, ldv, n, momentum, S, runs, W, s);
  else if (vec == 2) launch_step<2, kServer>(x, V, G, pv, ldv, n, momentum, S, runs, W, s);
  else launch_step<1, kServer>(x, V, G, pv, ldv, n, momentum, S, runs, W, s);
  return check_launch("nbsgd_step_server");
}

extern "C" nbsgd_status nbsgd_accumulate(const float* G, const uint8_t* mask, int32_t n, int32_t m,
                                         int64_t P, float* Gbar, void* stream) {
  clear_error();
  if (nbsgd_status st = check_nm(n, m)) return st;
  if (P < 0) return fail(NBSGD_E_SHAPE, "P=%lld is negative", (long long)P);
  Learners L;
  if (nbsgd_status st = learners_from_mask(mask, n, m, 1.0f, &L)) return st;
  if (P == 0) return NBSGD_OK;
  if (nbsgd_status st = check_rows(G, "G")) return st;
  if (nbsgd_status st = check_rows(Gbar, "Gbar")) return st;
  if (overlap(G, (int64_t)n * m * P * 4, Gbar, (int64_t)n * P * 4))
    return fail(NBSGD_E_ARG, "G and Gbar overlap");
  const int vec = vec_width(P);
  const int64_t pv = P / vec;
  const int64_t blocks = (pv + kBlock - 1) / kBlock;
  if (blocks > 0x7fffffff) return fail(NBSGD_E_UNSUPPORTED, "P too large");
  const dim3 grid((unsigned)blocks, (unsigned)n);
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  if (vec == 4) hipLaunchKernelGGL(k_accumulate<4>, grid, dim3(kBlock), 0, s, G, Gbar, pv, m, L);
  else if (vec == 2) hipLaunchKernelGGL(k_accumulate<2>, grid, dim3(kBlock), 0, s, G, Gbar, pv, m, L);
  else hipLaunchKernelGGL(k_accumulate<1>, grid, dim3(kBlock), 0, s, G, Gbar, pv, m, L);
  return check_launch("nbsgd_accumulate");
}

extern "C" nbsgd_status nbsgd_update(float* X, float* V, const float* Gbar, const int32_t* counts,
                                     int32_t n, int32_t m, int64_t P, float lr, float momentum,
                                     void* stream) {
  clear_error();
  if (nbsgd_status st = check_nm(n, m)) return st;
  if (P < 0) return fail(NBSGD_E_SHAPE, "P=%lld is negative", (long long)P);
  if (!counts) return fail(NBSGD_E_ARG, "counts is null");
  Learners L;
  memset(&L, 0, sizeof L);
  for (int32_t i = 0; i < n; ++i) {
    if (counts[i] < 1 || counts[i] > m)
      return fail(NBSGD_E_MASK, "counts[%d]=%d is outside [1, m=%d]", i, counts[i], m);
    L.eta[i] = (float)((double)lr * (double)counts[i] / (double)m);
  }
  if (P == 0) return NBSGD_OK;
  if (nbsgd_status st = check_rows(X, "X")) return st;
  if (nbsgd_status st = check_rows(V, "V")) return st;
  if (nbsgd_status st = check_rows(Gbar, "Gbar")) return st;
  const int64_t xb = (int64_t)n * P * 4;
  if (overlap(X, xb, V, xb) || overlap(X, xb, Gbar, xb) || overlap(V, xb, Gbar, xb))
    return fail(NBSGD_E_ARG, "X, V and Gbar must not overlap");
  const int vec = vec_width(P);
  const int64_t pv = P / vec;
  const int64_t blocks = (pv + kBlock - 1) / kBlock;
  if (blocks > 0x7fffffff) return fail(NBSGD_E_UNSUPPORTED, "P too large");
  const dim3 grid((unsigned)blocks, (unsigned)n);
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  if (vec == 4) hipLaunchKernelGGL(k_update<4>, grid, dim3(kBlock), 0, s, X, V, Gbar, pv, momentum, L);
  else if (vec == 2) hipLaunchKernelGGL(k_update<2>, grid, dim3(kBlock), 0, s, X, V, Gbar, pv, momentum, L);
  else hipLaunchKernelGGL(k_update<1>, grid, dim3(kBlock), 0, s, X, V, Gbar, pv, momentum, L);
  return check_launch("nbsgd_update");
}

extern "C" nbsgd_status nbsgd_mix(const float* X, const float* Wh, int32_t n, int64_t P, float* Y,
                                  void* stream) {
  clear_error();
  if (nbsgd_status st = check_nm(n, 1)) return st;
  if (P < 0) return fail(NBSGD_E_SHAPE, "P=%lld is negative", (long long)P);
  Mixing W;
  if (nbsgd_status st = mixing_from_w(Wh, n, &W)) return st;
  if (P == 0) return NBSGD_OK;
  if (nbsgd_status st = check_rows(X, "X")) return st;
  if (nbsgd_status st = check_rows(Y, "Y")) return st;
  const int64_t xb = (int64_t)n * P * 4;
  if (X != Y && overlap(X, xb, Y, xb)) return fail(NBSGD_E_ARG, "X and Y partially overlap");
  const int vec = vec_width(P);
  const int64_t pv = P / vec;
  const int64_t blocks = (pv + kWave - 1) / kWave;
  if (blocks > 0x7fffffff) return fail(NBSGD_E_UNSUPPORTED, "P too large");
  const size_t lds = (size_t)n * kWave * vec * sizeof(float);
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  if (vec == 4) hipLaunchKernelGGL(k_mix<4>, dim3((unsigned)blocks), dim3(kBlock), lds, s, X, Y, pv, n, W);
  else if (vec == 2) hipLaunchKernelGGL(k_mix<2>, dim3((unsigned)blocks), dim3(kBlock), lds, s, X, Y, pv, n, W);
  else hipLaunchKernelGGL(k_mix<1>, dim3((unsigned)blocks), dim3(kBlock), lds, s, X, Y, pv, n, W);
  return check_launch("nbsgd_mix");
}
