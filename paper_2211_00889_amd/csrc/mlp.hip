// End-to-end workload for gfx950: per-mini-batch gradients of a two-layer MLP
// (d_in -> hidden, ReLU -> classes, softmax cross-entropy, mean over a
// 32-sample mini-batch) written into G[i][j] of the Non-blocking step, and the
// mean loss of a parameter vector on a sample list (evaluation).
//
// Every GEMM input is rounded to bf16 (round to nearest even, the hardware
// conversion) and multiplied on the matrix cores with fp32 accumulation:
//   k_mlp_fwd    Z1 = A W1 (+ b1 in the head) MFMA 16x16x32, K = d_in in up to 4 ranges
//   k_mlp_head   H = relu(Z1), Z2 = H W2 + b2, softmax-CE, dZ2, dW2 = H^T dZ2,
//                db2, dH = dZ2 W2^T, dZ1 = dH * [Z1 > 0], db1   (N = classes
//                is below one 16-wide tile, so these run on the vector ALUs
//                with the same bf16-rounded inputs and fp32 sums)
//   k_mlp_wgrad  dW1 = A^T dZ1                MFMA 16x16x32, K = batch = 32
// MFMA 16x16x32 bf16 operand layout (lane l, t = 0..7): A[l % 16][8 (l / 16) + t],
// B[8 (l / 16) + t][l % 16]; result D[4 (l / 16) + t][l % 16], t = 0..3.
//
// Flat parameter layout of a replica: W1[d_in][hidden], b1[hidden],
// W2[hidden][classes], b2[classes].
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>
#include <string.h>

#include "internal.h"

using namespace nbsgd;

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

constexpr int kBatch = 32;       // mini-batch size (the MFMA K of dW1)
constexpr int kMaxHidden = 512;  // LDS of k_mlp_head
constexpr int kMaxClasses = 16;
constexpr int kMaxEntries = 512;  // mini-batches per launch (kernel-argument list)
constexpr int kIdxPerLaunch = 960;

struct Dims {
  int32_t d_in, hidden, classes;
  int64_t P;                     // parameters per replica
  int64_t off_b1, off_w2, off_b2;
};

// One launch's mini-batches: word k = (learner << 16) | slot.  The slot
// indexes the sample list (slot * 32 ..), the Z1/dZ1 workspace rows and the
// loss output; the learner selects the parameter row.
struct Entries {
  int32_t count;
  uint32_t e[kMaxEntries];
};

struct IdxChunk {
  int32_t v[kIdxPerLaunch];
};

__device__ __forceinline__ int entry_learner(uint32_t w) { return (int)(w >> 16); }
__device__ __forceinline__ int entry_slot(uint32_t w) { return (int)(w & 0xffffu); }

__device__ __forceinline__ float bf16r(float x) { return (float)(__bf16)x; }

__global__ void __launch_bounds__(256) k_put_idx(int32_t* __restrict__ dst, int32_t count, IdxChunk c) {
  const int t = blockIdx.x * 256 + threadIdx.x;
  if (t < count) dst[t] = c.v[t];
}

// Partial Z1: Z1p[z][slot][r][c] = sum over k in the z-th of gridDim.z equal
// K ranges of bf16(A[s_r][k]) bf16(W1[k][c]), for one mini-batch and 64
// hidden units; wave w owns 16 of them and all 32 rows.  Splitting K keeps
// more workgroups in flight; the loads of four 32-wide K steps are issued
// before their MFMAs.  The head kernel adds the partials (in z order) and b1.
__global__ void __launch_bounds__(256)
    k_mlp_fwd(const float* __restrict__ X, const float* __restrict__ data,
              const int32_t* __restrict__ idx, float* __restrict__ Z1p, int64_t part_stride,
              Dims d, Entries E) {
  constexpr int kU = 4;
  const uint32_t ew = E.e[blockIdx.y];
  const int slot = entry_slot(ew);
  const float* prm = X + (int64_t)entry_learner(ew) * d.P;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int col = blockIdx.x * 64 + wave * 16 + (lane & 15);
  const int kq = 8 * (lane >> 4);
  const int krange = d.d_in / (int)gridDim.z;
  const int kbeg = (int)blockIdx.z * krange;
  const float* a0 = data + (int64_t)idx[slot * kBatch + (lane & 15)] * d.d_in + kq;
  const float* a1 = data + (int64_t)idx[slot * kBatch + 16 + (lane & 15)] * d.d_in + kq;
  const float* w = prm + (int64_t)kq * d.hidden + col;
  f32x4 acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
  for (int k0 = kbeg; k0 < kbeg + krange; k0 += 32 * kU) {
    f32x4 x00[kU], x01[kU], x10[kU], x11[kU];
    float wb[kU][8];
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const int k = k0 + 32 * u;
      x00[u] = *reinterpret_cast<const f32x4*>(a0 + k);
      x01[u] = *reinterpret_cast<const f32x4*>(a0 + k + 4);
      x10[u] = *reinterpret_cast<const f32x4*>(a1 + k);
      x11[u] = *reinterpret_cast<const f32x4*>(a1 + k + 4);
#pragma unroll
      for (int t = 0; t < 8; ++t) wb[u][t] = w[(int64_t)(k + t) * d.hidden];
    }
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      bf16x8 fa0, fa1, fb;
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        fa0[t] = (__bf16)x00[u][t];
        fa0[t + 4] = (__bf16)x01[u][t];
        fa1[t] = (__bf16)x10[u][t];
        fa1[t + 4] = (__bf16)x11[u][t];
      }
#pragma unroll
      for (int t = 0; t < 8; ++t) fb[t] = (__bf16)wb[u][t];
      acc0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa0, fb, acc0, 0, 0, 0);
      acc1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa1, fb, acc1, 0, 0, 0);
    }
  }
  float* z = Z1p + (int64_t)blockIdx.z * part_stride + (int64_t)slot * kBatch * d.hidden + col;
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const int r = 4 * (lane >> 4) + t;
    z[(int64_t)r * d.hidden] = acc0[t];
    z[(int64_t)(r + 16) * d.hidden] = acc1[t];
  }
}

// Layer 2, the loss and (when BACKWARD) the layer-2 gradients, db1 and dZ1,
// one workgroup per mini-batch.
template <bool BACKWARD>
__global__ void __launch_bounds__(256)
    k_mlp_head(const float* __restrict__ X, const int32_t* __restrict__ labels,
               const int32_t* __restrict__ idx, float* __restrict__ Z1p, int64_t part_stride,
               int parts, float* __restrict__ dZ1, float* __restrict__ G, int64_t g_stride,
               float* __restrict__ losses, Dims d, Entries E) {
  __shared__ float Hs[kBatch * kMaxHidden];        // bf16(relu(Z1)), later dZ1
  __shared__ float W2s[kMaxHidden * kMaxClasses];  // bf16(W2)
  __shared__ float Zs[kBatch * kMaxClasses];       // logits, then dZ2
  __shared__ float Zb[kBatch * kMaxClasses];       // bf16(dZ2)
  __shared__ float row_loss[kBatch];
  __shared__ int ys[kBatch];
  const uint32_t ew = E.e[blockIdx.x];
  const int slot = entry_slot(ew);
  const int learner = entry_learner(ew);
  const float* prm = X + (int64_t)learner * d.P;
  const int H = d.hidden, C = d.classes;
  const int tid = threadIdx.x;
  float* z1 = Z1p + (int64_t)slot * kBatch * H;  // partial 0; receives the full Z1

  for (int k = tid; k < H * C; k += 256) W2s[k] = bf16r(prm[d.off_w2 + k]);
  for (int k = tid; k < kBatch * H; k += 256) {
    float z = z1[k];
    for (int q = 1; q < parts; ++q) z += z1[(int64_t)q * part_stride + k];
    z += prm[d.off_b1 + k % H];
    z1[k] = z;  // read back below by this same thread (same k -> o mapping)
    Hs[k] = bf16r(fmaxf(z, 0.0f));
  }
  if (tid < kBatch) {
    const int y = labels[idx[slot * kBatch + tid]];
    ys[tid] = y < 0 ? 0 : (y >= C ? C - 1 : y);
  }
  __syncthreads();
  for (int o = tid; o < kBatch * C; o += 256) {
    const int r = o / C, c = o % C;
    float acc = 0.0f;
    for (int h = 0; h < H; ++h) acc += Hs[r * H + h] * W2s[h * C + c];
    Zs[o] = acc + prm[d.off_b2 + c];
  }
  __syncthreads();
  if (tid < kBatch) {
    const int r = tid;
    float zmax = Zs[r * C];
    for (int c = 1; c < C; ++c) zmax = fmaxf(zmax, Zs[r * C + c]);
    float sum = 0.0f;
    for (int c = 0; c < C; ++c) sum += expf(Zs[r * C + c] - zmax);
    const float lse = zmax + logf(sum);
    row_loss[r] = lse - Zs[r * C + ys[r]];
    if (BACKWARD)
      for (int c = 0; c < C; ++c) {
        const float g = (expf(Zs[r * C + c] - lse) - (c == ys[r] ? 1.0f : 0.0f)) * (1.0f / kBatch);
        Zs[r * C + c] = g;
        Zb[r * C + c] = bf16r(g);
      }
  }
  __syncthreads();
  if (tid == 0) {
    float s = 0.0f;
    for (int r = 0; r < kBatch; ++r) s += row_loss[r];
    losses[slot] = s * (1.0f / kBatch);
  }
  if (!BACKWARD) return;
  float* g = G + (int64_t)slot * g_stride;
  if (tid < C) {
    float s = 0.0f;
    for (int r = 0; r < kBatch; ++r) s += Zs[r * C + tid];
    g[d.off_b2 + tid] = s;
  }
  for (int o = tid; o < H * C; o += 256) {  // dW2[h][c]
    const int h = o / C, c = o % C;
    float acc = 0.0f;
    for (int r = 0; r < kBatch; ++r) acc += Hs[r * H + h] * Zb[r * C + c];
    g[d.off_w2 + o] = acc;
  }
  __syncthreads();  // Hs is reused for dZ1 below
  float* dz = dZ1 + (int64_t)slot * kBatch * H;
  for (int o = tid; o < kBatch * H; o += 256) {  // dZ1[r][h]
    const int r = o / H, h = o % H;
    float acc = 0.0f;
    for (int c = 0; c < C; ++c) acc += Zb[r * C + c] * W2s[h * C + c];
    const float v = z1[o] > 0.0f ? acc : 0.0f;
    Hs[o] = v;
    dz[o] = v;
  }
  __syncthreads();
  for (int h = tid; h < H; h += 256) {  // db1[h]
    float s = 0.0f;
    for (int r = 0; r < kBatch; ++r) s += Hs[r * H + h];
    g[d.off_b1 + h] = s;
  }
}

// dW1[f][c] = sum_r bf16(A[s_r][f]) bf16(dZ1[r][c]) into G[slot]: a workgroup
// covers 64 features x 64 hidden units, wave w the features f0 + 16 w .. with
// one MFMA per 16x16 block.  The tile goes through LDS so that every store
// instruction writes 512 contiguous bytes (the MFMA result layout would give
// 64-byte pieces).  Stores are 8-byte vectors: a G row starts at slot * P
// floats and P may be only even, so 16-byte alignment is not guaranteed.
__global__ void __launch_bounds__(256)
    k_mlp_wgrad(const float* __restrict__ data, const int32_t* __restrict__ idx,
                const float* __restrict__ dZ1, float* __restrict__ G, int64_t g_stride, Dims d,
                Entries E) {
  constexpr int kLd = 64 + 4;  // padded LDS row
  __shared__ float tile[64 * kLd];
  const int slot = entry_slot(E.e[blockIdx.z]);
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int f0 = blockIdx.x * 64;
  const int c0 = blockIdx.y * 64;
  const int rq = 8 * (lane >> 4);
  bf16x8 fa;
#pragma unroll
  for (int t = 0; t < 8; ++t)
    fa[t] = (__bf16)data[(int64_t)idx[slot * kBatch + rq + t] * d.d_in + f0 + wave * 16 + (lane & 15)];
  const float* dz = dZ1 + (int64_t)slot * kBatch * d.hidden;
#pragma unroll
  for (int nb = 0; nb < 4; ++nb) {
    const int c = 16 * nb + (lane & 15);
    bf16x8 fb;
#pragma unroll
    for (int t = 0; t < 8; ++t) fb[t] = (__bf16)dz[(int64_t)(rq + t) * d.hidden + c0 + c];
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa, fb, acc, 0, 0, 0);
#pragma unroll
    for (int t = 0; t < 4; ++t) tile[(wave * 16 + 4 * (lane >> 4) + t) * kLd + c] = acc[t];
  }
  __syncthreads();
  float* g = G + (int64_t)slot * g_stride + (int64_t)f0 * d.hidden + c0;
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    const int e = q * 256 + threadIdx.x;  // 2048 float pairs of the 64 x 64 tile
    const int row = e >> 5, c2 = (e & 31) * 2;
    const f32x2 v = {tile[row * kLd + c2], tile[row * kLd + c2 + 1]};
    __builtin_nontemporal_store(v, reinterpret_cast<f32x2*>(g + (int64_t)row * d.hidden + c2));
  }
}

// ------------------------------------------------------------------ host

nbsgd_status check_shape(const nbsgd_mlp_shape* s, Dims* d) {
  if (!s) return fail(NBSGD_E_ARG, "shape is null");
  if (s->batch != kBatch)
    return fail(NBSGD_E_UNSUPPORTED, "batch=%d: only %d is supported", s->batch, kBatch);
  if (s->d_in < 128 || s->d_in % 128 || s->hidden < 64 || s->hidden % 64 || s->hidden > kMaxHidden)
    return fail(NBSGD_E_UNSUPPORTED,
                "d_in=%d must be a multiple of 128 and hidden=%d a multiple of 64, at most %d",
                s->d_in, s->hidden, kMaxHidden);
  if (s->classes < 2 || s->classes > kMaxClasses)
    return fail(NBSGD_E_UNSUPPORTED, "classes=%d must be in [2, %d]", s->classes, kMaxClasses);
  d->d_in = s->d_in;
  d->hidden = s->hidden;
  d->classes = s->classes;
  d->off_b1 = (int64_t)s->d_in * s->hidden;
  d->off_w2 = d->off_b1 + s->hidden;
  d->off_b2 = d->off_w2 + (int64_t)s->hidden * s->classes;
  d->P = d->off_b2 + s->classes;
  return NBSGD_OK;
}

constexpr int kMaxSplit = 4;

// K ranges of the forward GEMM: as many as possible up to 4, each a multiple
// of the 128-wide unrolled K step.
int k_split(const Dims& d) {
  for (int s = kMaxSplit; s > 1; s /= 2)
    if (d.d_in % (128 * s) == 0) return s;
  return 1;
}

size_t workspace_for(const Dims& d, int64_t rows) {
  // sample list, kMaxSplit partial Z1 planes and dZ1, each region 256-byte aligned
  auto up = [](size_t b) { return (b + 255) & ~(size_t)255; };
  return up((size_t)rows * 4) + (kMaxSplit + 1) * up((size_t)rows * d.hidden * 4);
}

struct Workspace {
  int32_t* idx;
  float* z1;           // kMaxSplit planes of [rows][hidden]
  int64_t z1_stride;   // floats between planes
  float* dz1;
};

Workspace carve(void* ws, const Dims& d, int64_t rows) {
  auto up = [](size_t b) { return (b + 255) & ~(size_t)255; };
  char* p = static_cast<char*>(ws);
  Workspace w;
  w.idx = reinterpret_cast<int32_t*>(p);
  p += up((size_t)rows * 4);
  w.z1 = reinterpret_cast<float*>(p);
  w.z1_stride = (int64_t)(up((size_t)rows * d.hidden * 4) / 4);
  p += kMaxSplit * up((size_t)rows * d.hidden * 4);
  w.dz1 = reinterpret_cast<float*>(p);
  return w;
}

nbsgd_status upload_idx(const int32_t* host, int64_t count, int64_t n_samples, int32_t* dst,
                        hipStream_t s) {
  for (int64_t k = 0; k < count; ++k)
    if (host[k] < 0 || host[k] >= n_samples)
      return fail(NBSGD_E_ARG, "sample index %d at position %lld is outside [0, %lld)", host[k],
                  (long long)k, (long long)n_samples);
  for (int64_t k0 = 0; k0 < count; k0 += kIdxPerLaunch) {
    IdxChunk c;
    const int32_t len = (int32_t)std::min<int64_t>(kIdxPerLaunch, count - k0);
    memcpy(c.v, host + k0, (size_t)len * 4);
    hipLaunchKernelGGL(k_put_idx, dim3((len + 255) / 256), dim3(256), 0, s, dst + k0, len, c);
  }
  return NBSGD_OK;
}

nbsgd_status launch_err(const char* what) {
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(NBSGD_E_HIP, "%s launch failed: %s", what, hipGetErrorString(e));
  return NBSGD_OK;
}

}  // namespace

extern "C" nbsgd_status nbsgd_mlp_param_count(const nbsgd_mlp_shape* s, int64_t* P) {
  clear_error();
  Dims d;
  if (nbsgd_status st = check_shape(s, &d)) return st;
  if (!P) return fail(NBSGD_E_ARG, "P is null");
  *P = d.P;
  return NBSGD_OK;
}

extern "C" nbsgd_status nbsgd_mlp_workspace_bytes(const nbsgd_mlp_shape* s, int64_t rows,
                                                  size_t* bytes) {
  clear_error();
  Dims d;
  if (nbsgd_status st = check_shape(s, &d)) return st;
  if (!bytes || rows < 0) return fail(NBSGD_E_ARG, "bytes is null or rows < 0");
  *bytes = workspace_for(d, rows);
  return NBSGD_OK;
}

extern "C" nbsgd_status nbsgd_mlp_grad(const float* X, int32_t n, int32_t m, const nbsgd_mlp_shape* s,
                                       const float* data, const int32_t* labels, int64_t n_samples,
                                       const int32_t* idx, const uint8_t* mask, float* G,
                                       float* losses, void* workspace, size_t workspace_bytes,
                                       void* stream) {
  clear_error();
  if (nbsgd_status st = check_nm(n, m)) return st;
  Dims d;
  if (nbsgd_status st = check_shape(s, &d)) return st;
  if (!X || !data || !labels || !idx || !mask || !G || !losses || !workspace)
    return fail(NBSGD_E_ARG, "null pointer argument");
  if (((uintptr_t)X | (uintptr_t)data | (uintptr_t)G | (uintptr_t)workspace) & 15)
    return fail(NBSGD_E_ALIGN, "X, data, G and workspace must be 16-byte aligned");
  if (n_samples < 1) return fail(NBSGD_E_SHAPE, "n_samples must be >= 1");
  const int64_t rows = (int64_t)n * m * kBatch;
  if (workspace_bytes < workspace_for(d, rows))
    return fail(NBSGD_E_ARG, "workspace of %zu bytes is below the %zu needed", workspace_bytes,
                workspace_for(d, rows));
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  const Workspace w = carve(workspace, d, rows);
  if (nbsgd_status r = upload_idx(idx, rows, n_samples, w.idx, st)) return r;
  const int64_t g_stride = d.P;  // G rows are [n][m][P]: slot i*m+j starts at slot*P
  Entries E;
  E.count = 0;
  auto flush = [&]() {
    if (E.count == 0) return;
    const int split = k_split(d);
    hipLaunchKernelGGL(k_mlp_fwd, dim3(d.hidden / 64, E.count, split), dim3(256), 0, st, X, data,
                       w.idx, w.z1, w.z1_stride, d, E);
    hipLaunchKernelGGL(k_mlp_head<true>, dim3(E.count), dim3(256), 0, st, X, labels, w.idx, w.z1,
                       w.z1_stride, split, w.dz1, G, g_stride, losses, d, E);
    hipLaunchKernelGGL(k_mlp_wgrad, dim3(d.d_in / 64, d.hidden / 64, E.count), dim3(256), 0, st,
                       data, w.idx, w.dz1, G, g_stride, d, E);
    E.count = 0;
  };
  for (int32_t i = 0; i < n; ++i)
    for (int32_t j = 0; j < m; ++j)
      if (mask[i * m + j]) {
        E.e[E.count++] = ((uint32_t)i << 16) | (uint32_t)(i * m + j);
        if (E.count == kMaxEntries) flush();
      }
  flush();
  return launch_err("nbsgd_mlp_grad");
}

extern "C" nbsgd_status nbsgd_mlp_loss(const float* params, const nbsgd_mlp_shape* s,
                                       const float* data, const int32_t* labels, int64_t n_samples,
                                       const int32_t* idx, int32_t count, float* losses,
                                       void* workspace, size_t workspace_bytes, void* stream) {
  clear_error();
  Dims d;
  if (nbsgd_status st = check_shape(s, &d)) return st;
  if (!params || !data || !labels || !idx || !losses || !workspace)
    return fail(NBSGD_E_ARG, "null pointer argument");
  if (((uintptr_t)params | (uintptr_t)data | (uintptr_t)workspace) & 15)
    return fail(NBSGD_E_ALIGN, "params, data and workspace must be 16-byte aligned");
  if (n_samples < 1) return fail(NBSGD_E_SHAPE, "n_samples must be >= 1");
  if (count < kBatch || count % kBatch || count / kBatch > kMaxEntries)
    return fail(NBSGD_E_SHAPE, "count=%d must be a multiple of %d, at most %d", count, kBatch,
                kBatch * kMaxEntries);
  if (workspace_bytes < workspace_for(d, count))
    return fail(NBSGD_E_ARG, "workspace of %zu bytes is below the %zu needed", workspace_bytes,
                workspace_for(d, count));
  Entries E;
  E.count = count / kBatch;
  for (int32_t k = 0; k < E.count; ++k) E.e[k] = (uint32_t)k;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  const Workspace w = carve(workspace, d, count);
  if (nbsgd_status r = upload_idx(idx, count, n_samples, w.idx, st)) return r;
  const int split = k_split(d);
  hipLaunchKernelGGL(k_mlp_fwd, dim3(d.hidden / 64, E.count, split), dim3(256), 0, st, params, data,
                     w.idx, w.z1, w.z1_stride, d, E);
  hipLaunchKernelGGL(k_mlp_head<false>, dim3(E.count), dim3(256), 0, st, params, labels, w.idx,
                     w.z1, w.z1_stride, split, w.dz1, nullptr, 0, losses, d, E);
  return launch_err("nbsgd_mlp_loss");
}
