// End-to-end workload for gfx950: per-mini-batch gradients of a two-layer MLP
// (d_in -> hidden, ReLU -> classes, softmax cross-entropy, mean over a
// 32-sample mini-batch) written into G[i][j] of the Non-blocking step, and the
// mean loss of a parameter vector on a sample list (evaluation).
//
// Every GEMM input is rounded to bf16 (round to nearest even, the hardware
// conversion) and multiplied with fp32 accumulation:
//   k_mlp_fwd_sk  partial Z1 = A W1 over one slice of d_in, per 128-row x
//                 128-unit tile, on MFMA 16x16x32 (both operands staged in LDS)
//   k_mlp_head    per mini-batch: Z1 = sum of the slices + b1, H =
//                 bf16(relu(Z1)), logits = H W2 + b2 (MFMA, classes padded to
//                 16), softmax-CE, dZ2; dZ1 = (dZ2 W2^T) * [Z1 > 0], db1, dW2 =
//                 H^T dZ2 (MFMA), db2 and the loss
//   k_mlp_wgrad  dW1 = A^T dZ1 on MFMA 16x16x32 (K = batch = 32), staged per
//                16-feature tile through LDS and stored as whole row pieces
// MFMA 16x16x32 bf16 operand layout (lane l, t = 0..7): A[l % 16][8 (l / 16) + t],
// B[8 (l / 16) + t][l % 16]; result D[4 (l / 16) + t][l % 16], t = 0..3.
//
// Flat parameter layout of a replica: W1[d_in][hidden], b1[hidden],
// W2[hidden][classes], b2[classes], then zeros up to a multiple of 4 floats,
// so every replica row and every G row starts 16-byte aligned (rows are ld
// floats apart, ld >= P a multiple of 4; ld = P unless the caller pads them).
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <vector>

#include "internal.h"
#include "mlp_shape.h"

using namespace nbsgd;

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// kBatch, kMaxHidden, kMaxClasses, kFeatBlock, kSkMaxSlices and Dims: mlp_shape.h
constexpr int kMaxList = 896;    // mini-batches per launch group (kernel-argument list)
constexpr int kMaxEval = 512;    // batches of 32 per nbsgd_mlp_loss call
constexpr int kHeadThreads = 1024;  // 16 waves per mini-batch in k_mlp_head

// One launch group's mini-batches, word e = learner << 24 | slot << 12,
// sorted by learner.  A slot indexes the caller's sample list (slot * 32 ..),
// the G rows and the loss output; the workspace rows of entry e are
// e * 32 .. e * 32 + 31.  Read as 32-bit words only.
struct List {
  int32_t count;
  uint32_t w[kMaxList];
};

// Sample indices of list entries first .. first + n_slots - 1, 32 per entry:
// two to a word (16 bits each) when `wide` is 0, one to a word otherwise.
constexpr int kUpSlots = 60;
struct IdxChunk {
  int32_t first, n_slots, wide;
  uint32_t v[kUpSlots * kBatch / 2];
};

// Sample indices of a whole launch group carried in the forward kernel's
// arguments (groups of at most kInline mini-batches whose indices all fit 16
// bits): row e * 32 + r in the 16-bit half r % 2 of word (e * 32 + r) / 2.
constexpr int kInline = 56;
template <int N>
struct Idx16 {
  uint32_t v[N];
};
using InlineIdx = Idx16<kInline * kBatch / 2>;

// kernel arguments are limited to 4 KiB: the list, the shapes and at most
// ten pointers or 64-bit scalars
static_assert(sizeof(List) + sizeof(Dims) + 10 * 8 <= 4096, "kernel arguments exceed 4 KiB");
static_assert(sizeof(IdxChunk) + 32 <= 4096, "kernel arguments exceed 4 KiB");
static_assert(kMaxList <= 4096 && kMaxEval <= 4096, "slots are packed in 16 bits");

__host__ __device__ __forceinline__ int item_learner(uint32_t w) { return (int)(w >> 24); }
__device__ __forceinline__ int item_slot(uint32_t w) { return (int)((w >> 12) & 0xfffu); }

__device__ __forceinline__ float bf16r(float x) { return (float)(__bf16)x; }

__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
  const __bf16 a = (__bf16)lo, b = (__bf16)hi;
  uint16_t ua, ub;
  __builtin_memcpy(&ua, &a, 2);
  __builtin_memcpy(&ub, &b, 2);
  return (uint32_t)ua | ((uint32_t)ub << 16);
}

// Writes the sample index of every row of the chunk's list entries (used
// when a group's indices do not fit the forward kernel's arguments).
__global__ void __launch_bounds__(256) k_put_idx(int32_t* __restrict__ dst, IdxChunk c) {
  const int t = blockIdx.x * 256 + threadIdx.x;
  if (t >= c.n_slots * kBatch) return;
  const int32_t v = c.wide ? (int32_t)c.v[t] : (int32_t)((c.v[t >> 1] >> (16 * (t & 1))) & 0xffffu);
  dst[c.first * kBatch + t] = v;
}

// Forward, split over d_in.  Work item: a quad (up to four mini-batches of one
// learner, 128 rows), a block of 128 hidden units and one of S equal slices of
// d_in (S = the largest divisor of d_in / 64 up to kSkMaxSlices).  Both operands
// are staged through LDS in bf16 ([row][k] and [unit][k]), so a 16-byte read
// is one MFMA fragment; the 16-byte k-octets of a row are XOR-swizzled so
// that the fragment reads and the staging writes are free of bank conflicts
// on gfx950 (A: 64 bf16 per row, octet o at o ^ (row % 8); W1: 80 bf16 per
// row, octet o at o ^ (unit / 4 % 8)).  Eight waves: wave w takes rows
// 32 (w % 4) .. +31 and units 64 (w / 4) .. +63 (2 x 4 accumulators).  The
// partial sums go to slice s of the partial buffer; k_mlp_head adds the
// slices in slice order.  The work items are split into eight equal ranges,
// one per XCD (workgroup b runs on XCD b % 8), so the items of one learner
// share an L2.  INLINE: the sample indices come from the kernel arguments and
// the workgroups of slice 0 and unit block 0 copy them to the workspace for
// the later kernels; otherwise they are read from the workspace.
constexpr int kSkRows = 128, kSkUnits = 128, kSkKc = 64, kSkLdA = kSkKc, kSkLdW = kSkKc + 16;
struct SkMap {
  int32_t n;              // learners present
  int32_t S;              // K slices
  int32_t ub;             // unit blocks
  uint32_t learner[4];    // learner id of present learner k in byte k % 4 of word k / 4
  int32_t off[17];        // first work item of each learner (off[n] = total)
  int32_t first[17];      // first list entry of each learner (first[n] = count)
};
static_assert(NBSGD_MAX_LEARNERS <= 16, "SkMap holds at most 16 learners");
static_assert(sizeof(InlineIdx) + sizeof(Dims) + sizeof(SkMap) + 5 * 8 <= 4096,
              "kernel arguments exceed 4 KiB");

template <bool INLINE>
__global__ void __launch_bounds__(512)
    k_mlp_fwd_sk(const float* __restrict__ X, const float* __restrict__ data,
                 int32_t* __restrict__ idx, float* __restrict__ Zpart, int64_t part_stride, Dims d,
                 SkMap M, Idx16<INLINE ? kInline * kBatch / 2 : 1> I) {
  constexpr int kDepth = 2;  // chunks loaded ahead of the one being staged
  __shared__ __attribute__((aligned(16))) __bf16 As[2][kSkRows * kSkLdA];
  __shared__ __attribute__((aligned(16))) __bf16 Ws[2][kSkUnits * kSkLdW];
  const int xcd = blockIdx.x & 7;
  const int64_t total = M.off[M.n];
  const int g = (int)(xcd * total / 8) + (int)(blockIdx.x >> 3);
  if (g >= (int)((xcd + 1) * total / 8)) return;  // uniform
  int li = 0;
  while (li + 1 < M.n && M.off[li + 1] <= g) ++li;
  const int cnt = M.first[li + 1] - M.first[li];
  const int quads = (cnt + 3) >> 2;
  int local = g - M.off[li];
  const int quad = local % quads;
  local /= quads;
  const int ubk = local % M.ub, s = local / M.ub;
  const int e0 = M.first[li] + 4 * quad;         // first list entry of the quad
  const int nmb = min(4, cnt - 4 * quad);
  const int rows = kBatch * nmb;
  const int H = d.hidden;
  const int u0 = kSkUnits * ubk;
  const int units = min(kSkUnits, H - u0);
  const int kslice = d.d_in / M.S, nck = kslice / kSkKc;
  const int kb = s * kslice;
  const int learner = (int)((M.learner[li >> 2] >> (8 * (li & 3))) & 0xffu);
  const float* prm = X + (int64_t)learner * d.ld;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wr = wave & 3, wu = wave >> 2;
  const bool mma = 32 * wr < rows && 64 * wu < units;  // wave-uniform

  // A staging: wave w takes rows 16 w .. +15, four consecutive lanes per row
  // (64 contiguous bytes, k = 4 q + 16 j + 0..3); the four rows of a 16-lane
  // group are two apart, which with the swizzle spreads its writes over all
  // banks.
  const int aquad = lane >> 2, aq = lane & 3;
  const int arow = 16 * wave + ((aquad >> 2) & 1) + 2 * (aquad & 3) + 8 * (aquad >> 3);
  // Rows past the tile's mini-batches read sample 0 and unit quads past the
  // block read its first units (both in bounds); stage() masks them to
  // zero.  The loads are unconditional, so the compiler can wait for one
  // register set while the next is still in flight.
  const bool alive = arow < rows;
  const float* asrc = data + kb + 4 * aq;
  if (alive) {
    const int t = e0 * kBatch + arow;  // workspace row: entry e0 + arow / 32, row arow % 32
    int32_t v;
    if constexpr (INLINE) {
      v = (int32_t)((I.v[t >> 1] >> (16 * (t & 1))) & 0xffffu);
      if (s == 0 && ubk == 0 && aq == 0) idx[t] = v;
    } else {
      v = idx[t];
    }
    asrc = data + (int64_t)v * d.d_in + kb + 4 * aq;
  }
  // W1 staging: k rows 4 wa .. +3, units 4 wq .. +3; wave w takes the k-quads
  // 2 w and 2 w + 1, four consecutive lanes read 64 contiguous bytes of one k
  // row, and each load of the wave reads two whole 512-byte row pieces.
  const int wa = 2 * wave + ((lane >> 2) & 1), wq = 4 * (lane >> 3) + (lane & 3);
  const bool wlive = 4 * wq < units;
  const float* wsrc = prm + (int64_t)(kb + 4 * wa) * H + u0 + 4 * (wlive ? wq : 0);
  // masks rather than selects, so the staging has no branches either
  const uint32_t amask = alive ? ~0u : 0u, wmask = wlive ? ~0u : 0u;

  struct Regs {
    f32x4 a[4], w[4];
  };
  auto load = [&](Regs& R, int c) {
    const int k0 = c * kSkKc;
#pragma unroll
    for (int j = 0; j < 4; ++j) R.a[j] = *reinterpret_cast<const f32x4*>(asrc + k0 + 16 * j);
#pragma unroll
    for (int r = 0; r < 4; ++r) R.w[r] = *reinterpret_cast<const f32x4*>(wsrc + (int64_t)(k0 + r) * H);
  };
  auto stage = [&](const Regs& R, int buf) {
    // k-quad aq + 4 j is half aq % 2 of octet aq / 2 + 2 j
    __bf16* a = As[buf] + arow * kSkLdA + 4 * (aq & 1);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint2 v = {pack_bf16(R.a[j][0], R.a[j][1]) & amask, pack_bf16(R.a[j][2], R.a[j][3]) & amask};
      *reinterpret_cast<uint2*>(a + 8 * (((aq >> 1) + 2 * j) ^ (arow & 7))) = v;
    }
    // units 4 wq + t, k-quad wa: half wa % 2 of octet wa / 2, swizzled by wq % 8
    __bf16* w = Ws[buf] + (4 * wq) * kSkLdW + 8 * ((wa >> 1) ^ (wq & 7)) + 4 * (wa & 1);
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const uint2 v = {pack_bf16(R.w[0][t], R.w[1][t]) & wmask, pack_bf16(R.w[2][t], R.w[3][t]) & wmask};
      *reinterpret_cast<uint2*>(w + t * kSkLdW) = v;
    }
  };
  f32x4 acc[2][4];
#pragma unroll
  for (int f = 0; f < 2; ++f)
#pragma unroll
    for (int u = 0; u < 4; ++u) acc[f][u] = f32x4{0.f, 0.f, 0.f, 0.f};
  auto multiply = [&](int buf) {
    if (!mma) return;
    // lane: row or unit l % 16 of the fragment, octet 4 ks + l / 16 (swizzled)
    const int g = lane >> 4;
    const __bf16* a = As[buf] + (32 * wr + (lane & 15)) * kSkLdA;
    const __bf16* w = Ws[buf] + (64 * wu + (lane & 15)) * kSkLdW;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const int oa = 8 * ((4 * ks + g) ^ (lane & 7));
      bf16x8 fa[2];
#pragma unroll
      for (int f = 0; f < 2; ++f)
        fa[f] = *reinterpret_cast<const bf16x8*>(a + 16 * f * kSkLdA + oa);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int ow = 8 * ((4 * ks + g) ^ (4 * (u & 1) + ((lane >> 2) & 3)));
        const bf16x8 fb = *reinterpret_cast<const bf16x8*>(w + 16 * u * kSkLdW + ow);
#pragma unroll
        for (int f = 0; f < 2; ++f)
          acc[f][u] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[f], fb, acc[f][u], 0, 0, 0);
      }
    }
  };
  // prologue: chunks 0 .. kDepth (indices clamped to the last chunk, so the
  // loads are unconditional and staging chunk 0 waits for its own loads only)
  Regs R[kDepth];
#pragma unroll
  for (int c = 0; c < kDepth; ++c) load(R[c], min(c, nck - 1));
  stage(R[0], 0);
  load(R[0], min(kDepth, nck - 1));
  __syncthreads();
  // step c: multiply chunk c (buffer c % 2); stage chunk c+1 from its register
  // set and refill that set with chunk c+1+kDepth
  auto step = [&](int c, Regs& Rn) {
    multiply(c & 1);
    if (c + 1 < nck) stage(Rn, (c + 1) & 1);
    if (c + 1 + kDepth < nck) load(Rn, c + 1 + kDepth);
    __syncthreads();
  };
  // steady state, branch-free: every step stages and refills its register set
  int c = 0;
  for (; c + 2 * kDepth < nck; c += kDepth) {
#pragma unroll
    for (int j = 0; j < kDepth; ++j) {
      multiply((c + j) & 1);
      stage(R[(j + 1) % kDepth], (c + j + 1) & 1);
      load(R[(j + 1) % kDepth], c + j + 1 + kDepth);
      __syncthreads();
    }
  }
  for (; c < nck; c += kDepth) {
#pragma unroll
    for (int j = 0; j < kDepth; ++j)
      if (c + j < nck) step(c + j, R[(j + 1) % kDepth]);
  }
  if (!mma) return;
  float* out = Zpart + (int64_t)s * part_stride;
#pragma unroll
  for (int f = 0; f < 2; ++f) {
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int r = 32 * wr + 16 * f + 4 * (lane >> 4) + t;
      if (r >= rows) continue;
      float* o = out + ((int64_t)e0 * kBatch + r) * H + u0 + 64 * wu + (lane & 15);
#pragma unroll
      for (int u = 0; u < 4; ++u) o[16 * u] = acc[f][u][t];
    }
  }
}

// Per list entry e = blockIdx.x (workspace rows e * 32 ..; G row and loss of
// its slot), all hidden units, 16 waves: the rows' labels (clamped into
// [0, classes)); Z1 = the S
// partial slices summed in slice order + b1 (kept in LDS); the logits =
// bf16(relu(Z1)) bf16(W2) + b2 on the matrix cores (classes zero-padded to
// 16; each wave takes every sixteenth 32-unit K step and the waves' partial
// sums are added in wave order); softmax cross-entropy, the loss and dZ2 =
// (softmax - onehot) / 32.  When BACKWARD, wave w takes the unit tiles
// 16 (w + 16 k) .. +15 on the matrix cores: dZ1 = (bf16(dZ2) bf16(W2)^T) *
// [Z1 > 0] (K = classes, zero-padded to 32), stored in bf16 as
// [entry][unit][row] for k_mlp_wgrad, db1 = its sum over the rows, and dW2 =
// bf16(relu(Z1))^T bf16(dZ2) (K = the 32 rows); then db2 and the padding of G.
template <bool BACKWARD>
__global__ void __launch_bounds__(kHeadThreads)
    k_mlp_head(const float* __restrict__ X, const int32_t* __restrict__ idx,
               const int32_t* __restrict__ labels, const float* __restrict__ Zpart,
               int64_t part_stride, int S,
               __bf16* __restrict__ dZ1t, float* __restrict__ G, float* __restrict__ losses, Dims d,
               List L) {
  constexpr int kLdz = kMaxHidden + 4;
  __shared__ __attribute__((aligned(16))) float Z1s[kBatch * kLdz];  // Z1 [row][unit]
  __shared__ float W2s[kMaxHidden * kMaxClasses];                     // bf16(W2), [unit][class]
  __shared__ float Zs[kBatch * kMaxClasses];  // logits, then dZ2
  __shared__ float Zb[kBatch * kMaxClasses];  // bf16(dZ2), zero beyond the classes
  __shared__ float row_loss[kBatch];
  __shared__ int ys[kBatch];
  __shared__ float Lp[(kHeadThreads / 64) * kBatch * 16];  // each wave's partial logits
  const uint32_t item = L.w[blockIdx.x];
  const int slot = item_slot(item);
  const float* prm = X + (int64_t)item_learner(item) * d.ld;
  const int H = d.hidden, C = d.classes;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t row0 = (int64_t)blockIdx.x * kBatch;
  const int32_t sample = tid < kBatch ? idx[row0 + tid] : 0;  // loaded ahead of its use

  // Z1: thread takes row tid / TPR and units uq + SPAN j, uq = 4 (tid % TPR).
  // Every load of this phase (the slices, b1, W2 and the label) is issued
  // before any of them is used, so the phase costs one memory round trip.
  constexpr int TPR = kHeadThreads / 32, SPAN = 4 * TPR;
  constexpr int kW2Loads = kMaxHidden * kMaxClasses / kHeadThreads;
  static_assert(4 * SPAN >= kMaxHidden && kW2Loads * kHeadThreads == kMaxHidden * kMaxClasses,
                "one pass of the phase covers every unit and every W2 entry");
  float b2v;  // b2 of class tid % 16, for the softmax thread (row tid / 16, class tid % 16)
  {
    const int r = tid / TPR, uq = 4 * (tid % TPR);
    const float* src = Zpart + (row0 + r) * H + uq;
    f32x4 p[kSkMaxSlices][4], b[4];
#pragma unroll
    for (int q = 0; q < kSkMaxSlices; ++q)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        p[q][j] = (q < S && uq + SPAN * j < H)
                      ? *reinterpret_cast<const f32x4*>(src + (int64_t)q * part_stride + SPAN * j)
                      : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < 4; ++j)
      b[j] = uq + SPAN * j < H ? *reinterpret_cast<const f32x4*>(prm + d.off_b1 + uq + SPAN * j)
                               : f32x4{0.f, 0.f, 0.f, 0.f};
    float w2[kW2Loads];
#pragma unroll
    for (int k = 0; k < kW2Loads; ++k) {
      const int e = tid + k * kHeadThreads;
      w2[k] = e < H * C ? prm[d.off_w2 + e] : 0.0f;
    }
    const int32_t y = tid < kBatch ? labels[sample] : 0;
    b2v = tid < kBatch * 16 && (tid & 15) < C ? prm[d.off_b2 + (tid & 15)] : 0.0f;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if (uq + SPAN * j >= H) break;
      f32x4 z = p[0][j];
#pragma unroll
      for (int q = 1; q < kSkMaxSlices; ++q)
        if (q < S) z += p[q][j];
      z += b[j];
      *reinterpret_cast<f32x4*>(Z1s + r * kLdz + uq + SPAN * j) = z;
    }
#pragma unroll
    for (int k = 0; k < kW2Loads; ++k) {
      const int e = tid + k * kHeadThreads;
      if (e < H * C) W2s[e] = bf16r(w2[k]);
    }
    if (tid < kBatch) ys[tid] = y < 0 ? 0 : (y >= C ? C - 1 : y);
  }
  __syncthreads();
  // logits = bf16(relu(Z1)) bf16(W2) on the matrix cores: wave w takes the
  // 32-unit K steps w, w + 16, .. for both 16-row tiles; the waves' partial
  // sums are added in wave order
  {
    const int kq8 = 8 * (lane >> 4), cl = lane & 15;
    f32x4 acc[2] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
    for (int ks = wave; ks < H / 32; ks += kHeadThreads / 64) {
      const int u0 = 32 * ks + kq8;
      bf16x8 fb;
#pragma unroll
      for (int t = 0; t < 8; ++t) fb[t] = (__bf16)(cl < C ? W2s[(u0 + t) * C + cl] : 0.0f);
#pragma unroll
      for (int rt = 0; rt < 2; ++rt) {
        const float* z = Z1s + (16 * rt + cl) * kLdz + u0;
        bf16x8 fa;
#pragma unroll
        for (int t = 0; t < 8; ++t) fa[t] = (__bf16)fmaxf(z[t], 0.0f);
        acc[rt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa, fb, acc[rt], 0, 0, 0);
      }
    }
    // lane holds rows 16 rt + 4 (lane / 16) + t of class cl
#pragma unroll
    for (int rt = 0; rt < 2; ++rt)
#pragma unroll
      for (int t = 0; t < 4; ++t)
        Lp[(wave * kBatch + 16 * rt + 4 * (lane >> 4) + t) * 16 + cl] = acc[rt][t];
  }
  __syncthreads();
  // softmax cross-entropy, thread (row tid / 16, class tid % 16): the logit
  // (the waves' partial sums in wave order, + b2), then the row's max and sum
  // of exponentials over the 16 lanes of the row by xor butterflies (every
  // lane of a row ends with the same sums)
  if (tid < kBatch * 16) {
    const int r = tid >> 4, c = tid & 15;
    const bool live = c < C;
    float z = 0.0f;
    for (int w = 0; w < kHeadThreads / 64; ++w) z += Lp[(w * kBatch + r) * 16 + c];
    z += b2v;
    float zmax = live ? z : -INFINITY;
#pragma unroll
    for (int o = 8; o; o >>= 1) zmax = fmaxf(zmax, __shfl_xor(zmax, o, 16));
    float sum = live ? expf(z - zmax) : 0.0f;
#pragma unroll
    for (int o = 8; o; o >>= 1) sum += __shfl_xor(sum, o, 16);
    const float lse = zmax + logf(sum);
    const int yr = ys[r];
    if (c == yr) row_loss[r] = lse - z;
    if (BACKWARD) {
      const float g = live ? (expf(z - lse) - (c == yr ? 1.0f : 0.0f)) * (1.0f / kBatch) : 0.0f;
      Zs[r * kMaxClasses + c] = g;
      Zb[r * kMaxClasses + c] = bf16r(g);
    }
  }
  __syncthreads();
  float* g = G + (int64_t)slot * d.ld;
  if (tid == 0) {
    float s = 0.0f;
    for (int r = 0; r < kBatch; ++r) s += row_loss[r];
    losses[slot] = s * (1.0f / kBatch);
  }
  if (!BACKWARD) return;
  if (tid < C) {
    float s = 0.0f;
    for (int r = 0; r < kBatch; ++r) s += Zs[r * kMaxClasses + tid];
    g[d.off_b2 + tid] = s;
  }
  if (tid < d.P - d.off_pad) g[d.off_pad + tid] = 0.0f;
  const int kq = 8 * (lane >> 4);  // this lane's K offset in a fragment
  bf16x8 fz[2];                    // A[r][k] = bf16(dZ2[r][k]), row tiles 0 and 1
#pragma unroll
  for (int rt = 0; rt < 2; ++rt)
#pragma unroll
    for (int t = 0; t < 8; ++t)
      fz[rt][t] = (__bf16)(kq + t < kMaxClasses ? Zb[(16 * rt + (lane & 15)) * kMaxClasses + kq + t] : 0.0f);
  for (int ut = wave; ut < H / 16; ut += kHeadThreads / 64) {
    const int hl = 16 * ut + (lane & 15);  // this lane's unit
    // dZ1 for rows 16 rt .. +15 and units 16 ut .. +15
    bf16x8 fw;  // B[k][h] = bf16(W2[h][k]), k = class
#pragma unroll
    for (int t = 0; t < 8; ++t) fw[t] = (__bf16)(kq + t < C ? W2s[hl * C + kq + t] : 0.0f);
    float db1 = 0.0f;
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fz[rt], fw, acc, 0, 0, 0);
      // lane holds rows 16 rt + 4 (lane / 16) + t of unit hl
      const int r0 = 16 * rt + 4 * (lane >> 4);
      float v[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        v[t] = Z1s[(r0 + t) * kLdz + hl] > 0.0f ? acc[t] : 0.0f;
        db1 += v[t];
      }
      const uint2 packed = {pack_bf16(v[0], v[1]), pack_bf16(v[2], v[3])};
      *reinterpret_cast<uint2*>(dZ1t + ((int64_t)blockIdx.x * H + hl) * kBatch + r0) = packed;
    }
    // db1: the four row groups of a unit sit in lanes l, l+16, l+32, l+48
    db1 += __shfl_xor(db1, 16);
    db1 += __shfl_xor(db1, 32);
    if (lane < 16) g[d.off_b1 + hl] = db1;
    // dW2[h][c] for units 16 ut .. +15: A[h][r] = bf16(relu(Z1[r][h])), B[r][c] = bf16(dZ2[r][c])
    bf16x8 fh, fd;
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      fh[t] = (__bf16)fmaxf(Z1s[(kq + t) * kLdz + hl], 0.0f);
      fd[t] = (__bf16)Zb[(kq + t) * kMaxClasses + (lane & 15)];
    }
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fh, fd, acc, 0, 0, 0);
    const int c = lane & 15;
    if (c < C) {
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int h = 16 * ut + 4 * (lane >> 4) + t;
        g[d.off_w2 + (int64_t)h * C + c] = acc[t];
      }
    }
  }
}

// dW1[f][h] = sum_r bf16(A[s_r][f]) bf16(dZ1[r][h]) for one list entry
// (blockIdx.x) and 128 features f0 .. f0+127 (blockIdx.y), every unit h.
// Computed transposed, D[h][f] = dZ1^T A: the A operand (8 rows r of one
// unit) is a 16-byte read of the [entry][unit][row] dZ1 copy, the B operand (8
// rows of one feature) comes from the sample rows staged transposed in LDS,
// and each lane's four results are consecutive units of one G row.  Wave w
// takes the hidden/64 consecutive unit tiles from w * hidden/64; per feature
// tile it passes its results through its own LDS rows and stores each
// feature's hidden/4 units as one contiguous piece; a workgroup writes 128
// whole G rows of dW1.
__global__ void __launch_bounds__(256)
    k_mlp_wgrad(const float* __restrict__ data, const int32_t* __restrict__ idx,
                const __bf16* __restrict__ dZ1t, float* __restrict__ G, Dims d, List L) {
  constexpr int kLda = kBatch + 8;  // bf16 per transposed sample column (16-byte aligned)
  __shared__ __attribute__((aligned(16))) __bf16 At[kFeatBlock * kLda];
  const int slot = item_slot(L.w[blockIdx.x]);
  const int f0 = blockIdx.y * kFeatBlock;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int H = d.hidden;
  const int64_t row0 = (int64_t)blockIdx.x * kBatch;
  // this wave's dZ1 fragments (hidden/64 <= 8 consecutive unit tiles),
  // loaded before the sample rows so both latencies overlap
  const __bf16* dz = dZ1t + row0 * H + 8 * (lane >> 4);  // [unit][row] of this mini-batch
  bf16x8 fa[kMaxHidden / 64];
  const int per = H / 64;  // unit tiles of this wave: wave * per .. + per - 1
#pragma unroll
  for (int u = 0; u < kMaxHidden / 64; ++u) {
    const int ht = wave * per + u;
    if (u < per) fa[u] = *reinterpret_cast<const bf16x8*>(dz + (int64_t)(16 * ht + (lane & 15)) * kBatch);
  }
  {
    // rows 2p, 2p+1 (p = tid / 16) of the mini-batch, features 4q .. 4q+3 and
    // 64 + 4q .. (q = tid % 16): packed pairs of rows into At[f][r].  A row
    // of At is four 16-byte pieces of 8 samples; piece c of feature f sits at
    // position c ^ ((f / 16) % 4), so that these writes (features four apart)
    // and the fragment reads both spread over all LDS banks.
    const int p = tid >> 4, q = 4 * (tid & 15);
    const int pw = 4 * ((p >> 2) ^ ((q >> 4) & 3)) + (p & 3);  // dword of row pair p
    const float* s0 = data + (int64_t)idx[row0 + 2 * p] * d.d_in + f0 + q;
    const float* s1 = data + (int64_t)idx[row0 + 2 * p + 1] * d.d_in + f0 + q;
    uint32_t* a32 = reinterpret_cast<uint32_t*>(At);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const f32x4 x0 = *reinterpret_cast<const f32x4*>(s0 + 64 * h);
      const f32x4 x1 = *reinterpret_cast<const f32x4*>(s1 + 64 * h);
#pragma unroll
      for (int t = 0; t < 4; ++t) a32[((64 * h + q + t) * kLda >> 1) + pw] = pack_bf16(x0[t], x1[t]);
    }
  }
  __syncthreads();
  bf16x8 fb[kFeatBlock / 16];
#pragma unroll
  for (int ft = 0; ft < kFeatBlock / 16; ++ft)
    fb[ft] = *reinterpret_cast<const bf16x8*>(
        &At[(16 * ft + (lane & 15)) * kLda + 8 * ((lane >> 4) ^ (ft & 3))]);
  // Per feature tile the wave's 16 features x 16 per units go through its own
  // LDS rows (pitch 16 kMaxHidden / 64 + 4 words, so the 16 features' 16-byte
  // writes fall on distinct banks), and are stored as whole 64 per-byte pieces
  // of each G row: 4 per lanes per row, 64 / (4 per) rows per store
  // (measured: 52.8 against 55.3 us with each store writing 64-byte pieces
  // of 16 rows straight from the accumulators).
  constexpr int kPitch = 16 * (kMaxHidden / 64) + 4;
  __shared__ __attribute__((aligned(16))) float Stg[4][16 * kPitch];
  float* st = Stg[wave];
  const int rowlanes = 4 * per;                 // lanes per feature row (16 B each)
  const int rows_per = 64 / rowlanes;           // feature rows per store instruction
  float* g = G + (int64_t)slot * d.ld + (int64_t)f0 * H + 16 * per * wave;
#pragma unroll
  for (int ft = 0; ft < kFeatBlock / 16; ++ft) {
#pragma unroll
    for (int u = 0; u < kMaxHidden / 64; ++u) {
      if (u >= per) break;
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[u], fb[ft], acc, 0, 0, 0);
      *reinterpret_cast<f32x4*>(st + (lane & 15) * kPitch + 16 * u + 4 * (lane >> 4)) = acc;
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    for (int r0 = 0; r0 < 16; r0 += rows_per) {
      const int fr = r0 + lane / rowlanes, cq = lane % rowlanes;
      if (lane < rows_per * rowlanes && fr < 16) {
        const f32x4 v = *reinterpret_cast<const f32x4*>(st + fr * kPitch + 4 * cq);
        *reinterpret_cast<f32x4*>(g + (int64_t)(16 * ft + fr) * H + 4 * cq) = v;
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }
}

// ------------------------------------------------------------------ host

struct Workspace {
  int32_t* idx;
  __bf16* dz1t;
  float* part;        // partial Z1 of each d_in slice
  int64_t part_stride;
};

Workspace carve(void* ws, const Dims& d, int64_t rows) {
  char* p = static_cast<char*>(ws);
  Workspace w;
  w.idx = reinterpret_cast<int32_t*>(p);
  p += up256((size_t)rows * 4);
  w.dz1t = reinterpret_cast<__bf16*>(p);
  p += up256((size_t)rows * d.hidden * 2);
  w.part = reinterpret_cast<float*>(p);
  w.part_stride = (int64_t)(up256((size_t)rows * d.hidden * 4) / 4);
  return w;
}

// Checks every sample index of the mini-batches `slots` (host idx[slot*32 ..]).
nbsgd_status check_idx(const int32_t* host, const int32_t* slots, int n_slots, int64_t n_samples) {
  for (int k = 0; k < n_slots; ++k)
    for (int r = 0; r < kBatch; ++r) {
      const int64_t pos = (int64_t)slots[k] * kBatch + r;
      if (host[pos] < 0 || host[pos] >= n_samples)
        return fail(NBSGD_E_ARG, "sample index %d at position %lld is outside [0, %lld)", host[pos],
                    (long long)pos, (long long)n_samples);
    }
  return NBSGD_OK;
}

// Copies the sample indices of list entries 0 .. count-1 (host idx[slot*32 ..]
// of entry e's slot mb[e].second) to the workspace rows e*32 .. through the
// kernel arguments of k_put_idx.
void put_idx(const int32_t* host, const std::pair<int, int>* mb, int count, bool wide,
             const Workspace& w, hipStream_t s) {
  const int per = wide ? kUpSlots / 2 : kUpSlots;
  for (int k0 = 0; k0 < count; k0 += per) {
    IdxChunk c;
    memset(&c, 0, sizeof(c));
    c.first = k0;
    c.n_slots = std::min(per, count - k0);
    c.wide = wide ? 1 : 0;
    for (int k = 0; k < c.n_slots; ++k) {
      const int32_t* src = host + (int64_t)mb[k0 + k].second * kBatch;
      for (int r = 0; r < kBatch; ++r) {
        const int t = k * kBatch + r;
        if (wide) c.v[t] = (uint32_t)src[r];
        else c.v[t >> 1] |= (uint32_t)src[r] << (16 * (t & 1));
      }
    }
    hipLaunchKernelGGL(k_put_idx, dim3((c.n_slots * kBatch + 255) / 256), dim3(256), 0, s, w.idx, c);
  }
}

nbsgd_status launch_err(const char* what) {
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(NBSGD_E_HIP, "%s launch failed: %s", what, hipGetErrorString(e));
  return NBSGD_OK;
}

uint32_t item(int learner, int slot) { return ((uint32_t)learner << 24) | ((uint32_t)slot << 12); }

// Launches the kernels over mini-batches `mb` (learner, slot), sorted by
// learner, of one group (at most kMaxList): the sample indices host_idx[slot
// * 32 ..] (checked) go to the workspace in the forward kernel's arguments
// when the group has at most kInline mini-batches and they fit 16 bits
// (`wide` false), otherwise through k_put_idx first.
template <bool BACKWARD>
void launch_group(const std::pair<int, int>* mb, int count, const int32_t* host_idx, bool wide,
                  const float* X, const float* data, const int32_t* labels, const Workspace& w,
                  float* G, float* losses, const Dims& d, hipStream_t st) {
  List items;
  items.count = count;
  for (int k = 0; k < count; ++k) items.w[k] = item(mb[k].first, mb[k].second);
  // forward over quads of each learner's mini-batches, slices of d_in
  SkMap K;
  memset(&K, 0, sizeof K);
  const int chunks = d.d_in / kSkKc;
  K.S = 1;
  for (int q = kSkMaxSlices; q >= 1; --q)
    if (chunks % q == 0) {
      K.S = q;
      break;
    }
  K.ub = (d.hidden + kSkUnits - 1) / kSkUnits;
  int sk_total = 0;
  for (int k = 0; k < items.count; ++k) {
    if (k == 0 || item_learner(items.w[k]) != item_learner(items.w[k - 1])) {
      if (K.n > 0) sk_total += K.S * K.ub * ((k - K.first[K.n - 1] + 3) / 4);
      K.off[K.n] = sk_total;
      K.first[K.n] = k;
      K.learner[K.n >> 2] |= (uint32_t)item_learner(items.w[k]) << (8 * (K.n & 3));
      ++K.n;
    }
  }
  sk_total += K.S * K.ub * ((items.count - K.first[K.n - 1] + 3) / 4);
  K.off[K.n] = sk_total;
  K.first[K.n] = items.count;
  // each XCD's range of work items holds at most ceil(total / 8)
  const dim3 fgrid(8 * ((sk_total + 7) / 8));
  if (!wide && count <= kInline) {
    InlineIdx I;
    memset(&I, 0, sizeof I);
    for (int e = 0; e < count; ++e) {
      const int32_t* src = host_idx + (int64_t)mb[e].second * kBatch;
      for (int r = 0; r < kBatch; ++r) {
        const int t = e * kBatch + r;
        I.v[t >> 1] |= (uint32_t)src[r] << (16 * (t & 1));
      }
    }
    hipLaunchKernelGGL(k_mlp_fwd_sk<true>, fgrid, dim3(512), 0, st, X, data, w.idx, w.part,
                       w.part_stride, d, K, I);
  } else {
    put_idx(host_idx, mb, count, wide, w, st);
    const Idx16<1> none = {{0u}};
    hipLaunchKernelGGL(k_mlp_fwd_sk<false>, fgrid, dim3(512), 0, st, X, data, w.idx, w.part,
                       w.part_stride, d, K, none);
  }
  hipLaunchKernelGGL(k_mlp_head<BACKWARD>, dim3(items.count), dim3(kHeadThreads), 0, st, X, w.idx,
                     labels, w.part, w.part_stride, K.S, w.dz1t, G, losses, d, items);
  if (BACKWARD)
    hipLaunchKernelGGL(k_mlp_wgrad, dim3(items.count, d.d_in / kFeatBlock), dim3(256), 0, st, data,
                       w.idx, w.dz1t, G, d, items);
}

}  // namespace

namespace {

// Argument checks shared by the gradient entry points, before the workspace
// and the sample indices (checked by the caller, in that order): shapes, row
// stride, pointers and alignment.  On success *d holds the shape with d->ld
// set and *finished the finished (learner * m + mini-batch) entries in order.
nbsgd_status mlp_grad_check(const float* X, int64_t ld, int32_t n, int32_t m,
                            const nbsgd_mlp_shape* s, const float* data, const int32_t* labels,
                            int64_t n_samples, const int32_t* idx, const uint8_t* mask, float* G,
                            float* losses, Dims* d, std::vector<int32_t>* finished) {
  if (nbsgd_status st = check_nm(n, m)) return st;
  if (nbsgd_status st = check_shape(s, d)) return st;
  if (ld == 0) ld = d->P;
  if (ld < d->P || ld % 4)
    return fail(NBSGD_E_SHAPE, "row stride %lld must be a multiple of 4 and at least P=%lld",
                (long long)ld, (long long)d->P);
  d->ld = ld;
  if (!X || !data || !labels || !idx || !mask || !G || !losses)
    return fail(NBSGD_E_ARG, "null pointer argument");
  if (((uintptr_t)X | (uintptr_t)data | (uintptr_t)G) & 15)
    return fail(NBSGD_E_ALIGN, "X, data and G must be 16-byte aligned");
  if (n_samples < 1) return fail(NBSGD_E_SHAPE, "n_samples must be >= 1");
  finished->clear();
  for (int32_t k = 0; k < n * m; ++k)
    if (mask[k]) finished->push_back(k);
  return NBSGD_OK;
}

// Launches the gradient kernels of the finished mini-batches in groups of at
// most kMaxList, each group's workspace rows starting at entry 0 of `w`.
nbsgd_status mlp_grad_launch(const float* X, int32_t m, const Dims& d, const float* data,
                             const int32_t* labels, int64_t n_samples, const int32_t* idx,
                             const std::vector<int32_t>& finished, float* G, float* losses,
                             const Workspace& w, hipStream_t st) {
  const bool wide = n_samples > 65536;
  std::pair<int, int> mb[kMaxList];
  int count = 0;
  for (int32_t k : finished) {
    mb[count++] = {k / m, k};
    if (count == kMaxList) {
      launch_group<true>(mb, count, idx, wide, X, data, labels, w, G, losses, d, st);
      count = 0;
    }
  }
  if (count) launch_group<true>(mb, count, idx, wide, X, data, labels, w, G, losses, d, st);
  return launch_err("nbsgd_mlp_grad");
}

nbsgd_status mlp_grad_impl(const float* X, int64_t ld, int32_t n, int32_t m,
                           const nbsgd_mlp_shape* s, const float* data, const int32_t* labels,
                           int64_t n_samples, const int32_t* idx, const uint8_t* mask, float* G,
                           float* losses, void* workspace, size_t workspace_bytes, void* stream) {
  Dims d;
  std::vector<int32_t> finished;
  if (nbsgd_status st = mlp_grad_check(X, ld, n, m, s, data, labels, n_samples, idx, mask, G,
                                       losses, &d, &finished))
    return st;
  if (!workspace) return fail(NBSGD_E_ARG, "null pointer argument");
  if ((uintptr_t)workspace & 15) return fail(NBSGD_E_ALIGN, "workspace must be 16-byte aligned");
  const int64_t rows = (int64_t)n * m * kBatch;
  if (workspace_bytes < workspace_for(d, rows))
    return fail(NBSGD_E_ARG, "workspace of %zu bytes is below the %zu needed", workspace_bytes,
                workspace_for(d, rows));
  if (nbsgd_status r = check_idx(idx, finished.data(), (int)finished.size(), n_samples)) return r;
  return mlp_grad_launch(X, m, d, data, labels, n_samples, idx, finished, G, losses,
                         carve(workspace, d, rows), reinterpret_cast<hipStream_t>(stream));
}

// ------------------------------------------------ allocation-free variant
// The workspace of nbsgd_mlp_grad_noalloc: a static device array, one copy
// per GPU the library is loaded on, held until the process ends.  Host code
// never passes `scratch` itself to a kernel (on the host the name is only a
// stand-in for the symbol): the device address of each GPU's copy comes from
// hipGetSymbolAddress with that GPU current, and is kept per device.
static __device__ __align__(256) unsigned char scratch[NBSGD_MLP_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of the current device's scratch, looked up once per device.
nbsgd_status scratch_address(hipStream_t stream, void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(NBSGD_E_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  if (stream) {
    hipDevice_t sdev = -1;
    e = hipStreamGetDevice(stream, &sdev);
    if (e != hipSuccess) return fail(NBSGD_E_HIP, "hipStreamGetDevice: %s", hipGetErrorString(e));
    if (sdev != dev)
      return fail(NBSGD_E_ARG, "stream belongs to device %d but device %d is current", (int)sdev,
                  dev);
  }
  if (dev < 0 || dev >= kMaxDevices)
    return fail(NBSGD_E_UNSUPPORTED, "device %d is beyond the %d devices supported", dev,
                kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(NBSGD_E_HIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev,
                  hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return NBSGD_OK;
}

}  // namespace

extern "C" nbsgd_status nbsgd_mlp_grad(const float* X, int32_t n, int32_t m, const nbsgd_mlp_shape* s,
                                       const float* data, const int32_t* labels, int64_t n_samples,
                                       const int32_t* idx, const uint8_t* mask, float* G,
                                       float* losses, void* workspace, size_t workspace_bytes,
                                       void* stream) {
  clear_error();
  return mlp_grad_impl(X, 0, n, m, s, data, labels, n_samples, idx, mask, G, losses, workspace,
                       workspace_bytes, stream);
}

extern "C" nbsgd_status nbsgd_mlp_grad_strided(const float* X, int64_t ld, int32_t n, int32_t m,
                                               const nbsgd_mlp_shape* s, const float* data,
                                               const int32_t* labels, int64_t n_samples,
                                               const int32_t* idx, const uint8_t* mask, float* G,
                                               float* losses, void* workspace,
                                               size_t workspace_bytes, void* stream) {
  clear_error();
  if (ld <= 0) return fail(NBSGD_E_SHAPE, "row stride %lld must be positive", (long long)ld);
  return mlp_grad_impl(X, ld, n, m, s, data, labels, n_samples, idx, mask, G, losses, workspace,
                       workspace_bytes, stream);
}

extern "C" nbsgd_status nbsgd_mlp_grad_noalloc(const float* X, int64_t ld, int32_t n, int32_t m,
                                               const nbsgd_mlp_shape* s, const float* data,
                                               const int32_t* labels, int64_t n_samples,
                                               const int32_t* idx, const uint8_t* mask, float* G,
                                               float* losses, void* stream) {
  clear_error();
  if (ld <= 0) return fail(NBSGD_E_SHAPE, "row stride %lld must be positive", (long long)ld);
  Dims d;
  std::vector<int32_t> finished;
  if (nbsgd_status st = mlp_grad_check(X, ld, n, m, s, data, labels, n_samples, idx, mask, G,
                                       losses, &d, &finished))
    return st;
  // workspace rows for one launch group: the kernels index them by the
  // group's list entries, so the largest group sets the size
  const int64_t rows = (int64_t)std::min<size_t>(finished.size(), kMaxList) * kBatch;
  const size_t need = workspace_for(d, rows);
  if (need > (size_t)NBSGD_MLP_SCRATCH_BYTES)
    return fail(NBSGD_E_UNSUPPORTED,
                "%zu finished mini-batches of this shape need %zu bytes of workspace, above the "
                "%zu-byte static scratch buffer (use nbsgd_mlp_grad_strided with a workspace)",
                finished.size(), need, (size_t)NBSGD_MLP_SCRATCH_BYTES);
  if (nbsgd_status r = check_idx(idx, finished.data(), (int)finished.size(), n_samples)) return r;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  void* ws = nullptr;
  if (nbsgd_status r = scratch_address(st, &ws)) return r;
  return mlp_grad_launch(X, m, d, data, labels, n_samples, idx, finished, G, losses,
                         carve(ws, d, rows), st);
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
  if (count < kBatch || count % kBatch || count / kBatch > kMaxEval)
    return fail(NBSGD_E_SHAPE, "count=%d must be a multiple of %d, at most %d", count, kBatch,
                kBatch * kMaxEval);
  if (workspace_bytes < workspace_for(d, count))
    return fail(NBSGD_E_ARG, "workspace of %zu bytes is below the %zu needed", workspace_bytes,
                workspace_for(d, count));
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  const Workspace w = carve(workspace, d, count);
  std::pair<int, int> mb[kMaxEval];
  int32_t slots[kMaxEval];
  for (int32_t k = 0; k < count / kBatch; ++k) {
    mb[k] = {0, k};
    slots[k] = k;
  }
  if (nbsgd_status r = check_idx(idx, slots, count / kBatch, n_samples)) return r;
  launch_group<false>(mb, count / kBatch, idx, n_samples > 65536, params, data, labels, w, nullptr,
                      losses, d, st);
  return launch_err("nbsgd_mlp_loss");
}
