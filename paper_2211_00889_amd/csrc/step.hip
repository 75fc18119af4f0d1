// Device half of libnbsgd for gfx950: the fused Non-blocking step and its three
// unfused stages (accumulate, mix, update), with their argument checks.
//
// Data layout (all fp32, row-major, caller-owned HBM):
//   X, V  [n][P]      replicas and momentum buffers, learner-major
//   G     [n][m][P]   per-mini-batch gradients
// Every kernel works on column tiles: the mix couples learners, never
// columns, so a workgroup that holds all n rows of its columns can update X in
// place.  Rows are streamed as VEC-wide vectors (VEC = 4 when P % 4 == 0, else
// 2 or 1), so each wave moves 64 * VEC * 4 contiguous bytes per row per load.
//
// Fused step, one workgroup = 4 waves x (64 lanes * U vectors) columns:
//   phase 1: wave w takes learners p = w, w+4, ...; for its columns it reads
//            X[p], V[p] and only the finished rows of G[p], forms the new
//            momentum (stored at once) and the value to be mixed, z_p = x_p
//            (mix-then-step) or x_p - eta_p v_p (step-then-mix), into LDS;
//   phase 2: after one barrier, wave w forms row i = w, w+4, ... of the mix
//            from LDS (CSR of the nonzero W entries, or one sum scaled by 1/n
//            for uniform W) and writes X[i].
// HBM traffic per step is the finished rows of G once, X and V read once and
// written once: 4 * P * (sum_i c_i + 4 n) bytes.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>
#include <string.h>

#include "internal.h"

using namespace nbsgd;

namespace {

constexpr int kWave = 64;
constexpr int kWaves = 4;
constexpr int kBlock = kWave * kWaves;
constexpr int kMaxN = NBSGD_MAX_LEARNERS;
constexpr int kMaxM = NBSGD_MAX_MINIBATCHES;
constexpr int kSlots = (kMaxN + kWaves - 1) / kWaves;  // learners per wave

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

// Per-learner constants of one step, passed by value in the kernel arguments.
struct Learners {
  float eta[kMaxN];           // lr * c_i / m
  float inv_c[kMaxN];         // 1 / c_i
  int32_t count[kMaxN];       // c_i
  // indices of the finished mini-batches, four 8-bit indices per word so the
  // kernel reads them with scalar loads
  uint32_t rows[kMaxN][kMaxM / 4];
};

__device__ __forceinline__ int row_of(const Learners& L, int p, int r) {
  return (int)((L.rows[p][r >> 2] >> (8 * (r & 3))) & 0xffu);
}

// Mixing matrix as CSR over its nonzero entries, or the uniform flag.
struct Mixing {
  int32_t uniform;   // all entries equal: out = (sum_p z_p) * w_all
  float w_all;
  int32_t start[kMaxN + 1];
  uint8_t col[kMaxN * kMaxN];
  float w[kMaxN * kMaxN];
};

template <typename T>
__device__ __forceinline__ T ld_stream(const T* p) {
  return __builtin_nontemporal_load(p);
}
template <typename T>
__device__ __forceinline__ void st_stream(T* p, T v) {
  __builtin_nontemporal_store(v, p);
}

// Sum of the finished rows of learner p at vector column v.
template <int VEC>
__device__ __forceinline__ typename Vec<VEC>::type finished_sum(const typename Vec<VEC>::type* G,
                                                                const Learners& L, int p, int m,
                                                                int64_t pv, int64_t v) {
  using vf = typename Vec<VEC>::type;
  const vf* g = G + (int64_t)p * m * pv + v;
  const int c = L.count[p];
  vf acc = (vf)(0.0f);
  int r = 0;
  for (; r + 4 <= c; r += 4) {
    const uint32_t w = L.rows[p][r >> 2];
    const vf a0 = ld_stream(g + (int64_t)(w & 0xffu) * pv);
    const vf a1 = ld_stream(g + (int64_t)((w >> 8) & 0xffu) * pv);
    const vf a2 = ld_stream(g + (int64_t)((w >> 16) & 0xffu) * pv);
    const vf a3 = ld_stream(g + (int64_t)(w >> 24) * pv);
    acc += (a0 + a1) + (a2 + a3);
  }
  const int rem = c - r;  // 0..3 rows left, loaded together
  if (rem > 0) {
    const vf a0 = ld_stream(g + (int64_t)row_of(L, p, r) * pv);
    vf a1 = (vf)(0.0f), a2 = (vf)(0.0f);
    if (rem > 1) a1 = ld_stream(g + (int64_t)row_of(L, p, r + 1) * pv);
    if (rem > 2) a2 = ld_stream(g + (int64_t)row_of(L, p, r + 2) * pv);
    acc += (a0 + a1) + a2;
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
  for (int e = W.start[i]; e < W.start[i + 1]; ++e) acc += W.w[e] * zs[W.col[e] * ncols + t];
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

template <int VEC, int U, int ORDER>
__global__ void __launch_bounds__(kBlock)
    k_step(float* __restrict__ Xf, float* __restrict__ Vf, const float* __restrict__ Gf,
           int64_t pv, int n, int m, float mu, Learners L, Mixing W) {
  using vf = typename Vec<VEC>::type;
  extern __shared__ char smem[];
  vf* zs = reinterpret_cast<vf*>(smem);  // [n][U * 64]
  constexpr int ncols = U * kWave;
  vf* X = reinterpret_cast<vf*>(Xf);
  vf* V = reinterpret_cast<vf*>(Vf);
  const vf* G = reinterpret_cast<const vf*>(Gf);

  const int lane = threadIdx.x & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const int64_t col0 = (int64_t)blockIdx.x * ncols;

  vf keep[kSlots][U];  // eta_i * v_i for mix-then-step
#pragma unroll
  for (int s = 0; s < kSlots; ++s) {
    const int p = wave + kWaves * s;
    if (p < n) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int t = lane + kWave * u;
        const int64_t v = col0 + t;
        if (v < pv) {
          const int64_t off = (int64_t)p * pv + v;
          const vf x = ld_stream(X + off);
          const vf vo = ld_stream(V + off);
          const vf g = finished_sum<VEC>(G, L, p, m, pv, v);
          const vf vn = mu * vo + g * L.inv_c[p];
          st_stream(V + off, vn);
          if (ORDER == NBSGD_MIX_THEN_STEP) {
            zs[p * ncols + t] = x;
            keep[s][u] = L.eta[p] * vn;
          } else {
            zs[p * ncols + t] = x - L.eta[p] * vn;
          }
        }
      }
    }
  }
  __syncthreads();
  vf total[U];
  if (W.uniform) {
#pragma unroll
    for (int u = 0; u < U; ++u) total[u] = mix_all<VEC>(zs, ncols, n, lane + kWave * u) * W.w_all;
  }
#pragma unroll
  for (int s = 0; s < kSlots; ++s) {
    const int i = wave + kWaves * s;
    if (i < n) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int t = lane + kWave * u;
        const int64_t v = col0 + t;
        if (v < pv) {
          vf x = W.uniform ? total[u] : mix_row<VEC>(zs, ncols, W, i, t);
          if (ORDER == NBSGD_MIX_THEN_STEP) x -= keep[s][u];
          st_stream(X + (int64_t)i * pv + v, x);
        }
      }
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

nbsgd_status learners_from_mask(const uint8_t* mask, int32_t n, int32_t m, float lr, Learners* L) {
  if (!mask) return fail(NBSGD_E_ARG, "mask is null");
  memset(L, 0, sizeof *L);
  for (int32_t i = 0; i < n; ++i) {
    int32_t c = 0;
    for (int32_t j = 0; j < m; ++j)
      if (mask[i * m + j]) {
        L->rows[i][c >> 2] |= (uint32_t)j << (8 * (c & 3));
        ++c;
      }
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
        W->col[e] = (uint8_t)p;
        W->w[e] = Wh[i * n + p];
        ++e;
      }
  }
  W->start[n] = e;
  return NBSGD_OK;
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

constexpr int kStepU = 1;

template <int VEC, int ORDER>
void launch_step(float* X, float* V, const float* G, int64_t pv, int n, int m, float mu,
                 const Learners& L, const Mixing& W, hipStream_t s) {
  constexpr int ncols = kStepU * kWave;
  const int64_t blocks = (pv + ncols - 1) / ncols;
  const size_t lds = (size_t)n * ncols * VEC * sizeof(float);
  hipLaunchKernelGGL((k_step<VEC, kStepU, ORDER>), dim3((unsigned)blocks), dim3(kBlock), lds, s, X,
                     V, G, pv, n, m, mu, L, W);
}

}  // namespace

extern "C" nbsgd_status nbsgd_step(float* X, float* V, const float* G, const uint8_t* mask,
                                   const float* Wh, int32_t n, int32_t m, int64_t P, float lr,
                                   float momentum, int32_t order, void* stream) {
  clear_error();
  if (nbsgd_status st = check_nm(n, m)) return st;
  if (P < 0) return fail(NBSGD_E_SHAPE, "P=%lld is negative", (long long)P);
  if (order != NBSGD_MIX_THEN_STEP && order != NBSGD_STEP_THEN_MIX)
    return fail(NBSGD_E_ARG, "unknown order %d", order);
  Learners L;
  if (nbsgd_status st = learners_from_mask(mask, n, m, lr, &L)) return st;
  Mixing W;
  if (nbsgd_status st = mixing_from_w(Wh, n, &W)) return st;
  if (P == 0) return NBSGD_OK;
  if (nbsgd_status st = check_rows(X, "X")) return st;
  if (nbsgd_status st = check_rows(V, "V")) return st;
  if (nbsgd_status st = check_rows(G, "G")) return st;
  const int64_t xb = (int64_t)n * P * 4, gb = (int64_t)n * m * P * 4;
  if (overlap(X, xb, V, xb)) return fail(NBSGD_E_ARG, "X and V overlap");
  if (overlap(G, gb, X, xb) || overlap(G, gb, V, xb))
    return fail(NBSGD_E_ARG, "G overlaps X or V");
  const int vec = vec_width(P);
  const int64_t pv = P / vec;
  if ((pv + kStepU * kWave - 1) / (kStepU * kWave) > 0x7fffffff)
    return fail(NBSGD_E_UNSUPPORTED, "P=%lld needs too many workgroups", (long long)P);
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  if (order == NBSGD_MIX_THEN_STEP) {
    if (vec == 4) launch_step<4, NBSGD_MIX_THEN_STEP>(X, V, G, pv, n, m, momentum, L, W, s);
    else if (vec == 2) launch_step<2, NBSGD_MIX_THEN_STEP>(X, V, G, pv, n, m, momentum, L, W, s);
    else launch_step<1, NBSGD_MIX_THEN_STEP>(X, V, G, pv, n, m, momentum, L, W, s);
  } else {
    if (vec == 4) launch_step<4, NBSGD_STEP_THEN_MIX>(X, V, G, pv, n, m, momentum, L, W, s);
    else if (vec == 2) launch_step<2, NBSGD_STEP_THEN_MIX>(X, V, G, pv, n, m, momentum, L, W, s);
    else launch_step<1, NBSGD_STEP_THEN_MIX>(X, V, G, pv, n, m, momentum, L, W, s);
  }
  return check_launch("nbsgd_step");
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
