// End-to-end workload for gfx950: per-mini-batch gradients of a two-layer MLP
// (d_in -> hidden, ReLU -> classes, softmax cross-entropy, mean over a
// 32-sample mini-batch) written into G[i][j] of the Non-blocking step, and the
// mean loss of a parameter vector on a sample list (evaluation).
//
// Every GEMM input is rounded to bf16 (round to nearest even, the hardware
// conversion) and multiplied with fp32 accumulation:
//   k_mlp_fwd    Z1 = A W1 + b1 on MFMA 16x16x32 (full K per tile), then in
//                the epilogue H = bf16(relu(Z1)) and this tile's 64-unit share
//                of the logits, sum_h H W2 (vector ALUs; N = classes is below
//                one 16-wide MFMA tile)
//   k_mlp_head   logits = sum of the shares + b2, softmax-CE, dZ2; per 64
//                hidden units dW2 = H^T dZ2, dZ1 = (dZ2 W2^T) * [Z1 > 0], db1;
//                db2 and the loss once per mini-batch
//   k_mlp_wgrad  dW1 = A^T dZ1 on MFMA 16x16x32 (K = batch = 32), each lane
//                storing four consecutive hidden units of one G row
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
#include <vector>

#include "internal.h"

using namespace nbsgd;

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kBatch = 32;       // mini-batch size (the MFMA K of dW1)
constexpr int kMaxHidden = 512;
constexpr int kMaxClasses = 16;  // the logit shares are stored 16 wide
constexpr int kMaxList = 896;    // mini-batches per launch (kernel-argument list)
constexpr int kMaxEval = 512;    // batches of 32 per nbsgd_mlp_loss call
constexpr int kFeatBlock = 128;  // d_in features per k_mlp_wgrad workgroup

struct Dims {
  int32_t d_in, hidden, classes;
  int64_t P;                     // padded parameters per replica
  int64_t ld;                    // floats from one row of X (and of G) to the next, >= P
  int64_t off_b1, off_w2, off_b2, off_pad;
};

// One launch's work items, word k = learner << 24 | slot_a << 12 | (slot_b + 1).
// A slot indexes the sample list (slot * 32 ..), the workspace rows and the
// loss output; k_mlp_fwd takes up to two mini-batches of one learner per item
// (slot_b + 1 == 0: one), the other kernels one.  Read as 32-bit words only.
struct List {
  int32_t count;
  uint32_t w[kMaxList];
};

// Sample indices of up to kUpSlots mini-batches: word k of `slot` holds
// slots 2k and 2k+1 (16 bits each); `v` holds 32 indices per slot, two to a
// word (16 bits each) when `wide` is 0, one to a word otherwise.
constexpr int kUpSlots = 60;
struct IdxChunk {
  int32_t n_slots, wide;
  uint32_t slot[kUpSlots / 2];
  uint32_t v[kUpSlots * kBatch / 2];
};

// kernel arguments are limited to 4 KiB: the list, the shapes, the forward
// map and at most ten pointers or 64-bit scalars
static_assert(sizeof(List) + sizeof(Dims) + 180 + 10 * 8 <= 4096, "kernel arguments exceed 4 KiB");
static_assert(sizeof(IdxChunk) + 32 <= 4096, "kernel arguments exceed 4 KiB");
static_assert(kMaxList <= 4096 && kMaxEval <= 4096, "slots are packed in 16 bits");

__device__ __forceinline__ int item_learner(uint32_t w) { return (int)(w >> 24); }
__device__ __forceinline__ int item_slot_a(uint32_t w) { return (int)((w >> 12) & 0xfffu); }
__device__ __forceinline__ int item_slot_b(uint32_t w) { return (int)(w & 0xfffu) - 1; }

__device__ __forceinline__ float bf16r(float x) { return (float)(__bf16)x; }

__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
  const __bf16 a = (__bf16)lo, b = (__bf16)hi;
  uint16_t ua, ub;
  __builtin_memcpy(&ua, &a, 2);
  __builtin_memcpy(&ub, &b, 2);
  return (uint32_t)ua | ((uint32_t)ub << 16);
}

// Writes the sample index and its label (clamped into [0, classes)) of every
// row of the listed mini-batches.
__global__ void __launch_bounds__(256)
    k_put_idx(int32_t* __restrict__ dst, int32_t* __restrict__ ylab,
              const int32_t* __restrict__ labels, int32_t classes, IdxChunk c) {
  const int t = blockIdx.x * 256 + threadIdx.x;
  const int k = t >> 5, r = t & 31;
  if (k >= c.n_slots) return;
  const int slot = (int)((c.slot[k >> 1] >> (16 * (k & 1))) & 0xffffu);
  const int32_t v = c.wide ? (int32_t)c.v[t] : (int32_t)((c.v[t >> 1] >> (16 * (t & 1))) & 0xffffu);
  const int32_t y = labels[v];
  dst[slot * kBatch + r] = v;
  ylab[slot * kBatch + r] = y < 0 ? 0 : (y >= classes ? classes - 1 : y);
}

// Forward work items: the (tile, 64-unit block) pairs in order learner,
// unit block, tile, cut into 8 contiguous ranges, one per XCD (workgroup b
// runs on XCD b % 8), so the workgroups that share a tile's sample rows or a
// learner's W1 block share one L2.  Item g of learner i is unit block
// (g - off[i]) / tiles_i of tile first[i] + (g - off[i]) % tiles_i.
struct FwdMap {
  int32_t n;                // learners present
  int32_t xcd_start[9];     // item range of each XCD
  int32_t off[17];          // first item of each learner (off[n] = total)
  int32_t first[17];        // first tile of each learner in the tile list
};
static_assert(sizeof(FwdMap) <= 180, "forward map grew: recheck the kernel-argument budget");

// Z1 for up to 64 rows (the mini-batches slot_a, slot_b of one learner) and
// the 64 hidden units c0 .. c0+63, over the whole of d_in.  Eight waves:
// wave w takes rows 16 (w % 4) .. +15, all 64 units (four 16x16
// accumulators) and the K half w / 4 (64-deep chunks h, h+2, ...); its A
// fragments come straight from the sample rows.  Each half stages its W1
// chunks through LDS, transposed to [unit][k] in bf16 so that a B fragment
// is one 16-byte read.  Loads run two chunks ahead: while chunk s is
// multiplied, chunk s+1 is in LDS-bound registers and s+2 in flight.  The
// halves' sums are added in half order.  Epilogue: Z1 (+ b1) to the
// workspace, then this tile's share of the logits Zp[block][row][c] = sum
// over its 64 units of bf16(relu(Z1)) bf16(W2).
__global__ void __launch_bounds__(512)
    k_mlp_fwd(const float* __restrict__ X, const float* __restrict__ data,
              const int32_t* __restrict__ idx, float* __restrict__ Z1, float* __restrict__ Zp,
              int64_t zp_stride, Dims d, FwdMap M, List L) {
  constexpr int kKc = 64;        // K per staged chunk
  constexpr int kDepth = 2;      // chunks loaded ahead of the one being staged
  constexpr int kLdb = kKc + 8;  // bf16 per transposed row (16-byte aligned, padded)
  constexpr int kLdh = 64 + 1;
  constexpr int kLdp = 64 + 1;   // padded partial-sum row
  constexpr int kStage = 64 * kLdb;  // bf16 per staging buffer
  // 2 halves x 2 buffers of staging; after the K loop it holds half 1's sums
  __shared__ __attribute__((aligned(16))) __bf16 Bs[2 * 2 * kStage];
  __shared__ float Hs[64 * kLdh];
  __shared__ float W2s[64 * kMaxClasses];
  static_assert(64 * kLdp * 4 <= (int)sizeof(Bs), "partial sums exceed the staging space");
  const int xcd = blockIdx.x & 7;
  const int g = M.xcd_start[xcd] + (int)(blockIdx.x >> 3);
  if (g >= M.xcd_start[xcd + 1]) return;  // uniform: the whole workgroup leaves
  int li = 0;
  while (li + 1 < M.n && M.off[li + 1] <= g) ++li;
  const int tiles_i = (M.off[li + 1] - M.off[li]) / (d.hidden / 64);
  const int c0 = 64 * ((g - M.off[li]) / tiles_i);
  const uint32_t item = L.w[M.first[li] + (g - M.off[li]) % tiles_i];
  const int slot_a = item_slot_a(item), slot_b = item_slot_b(item);
  const int rows = slot_b >= 0 ? 64 : 32;
  const float* prm = X + (int64_t)item_learner(item) * d.ld;
  const int H = d.hidden, C = d.classes;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int half = wave >> 2, wr = wave & 3;
  const int htid = tid & 255;  // thread index within the half
  const bool mma = 16 * wr < rows;  // wave-uniform
  // W1 staging: rows 4a .. 4a+3 of the chunk, units 4q .. 4q+3 (each load
  // instruction reads whole 256-byte row pieces)
  const int sa = htid >> 4, sq = 4 * (htid & 15);
  const float* wsrc = prm + (int64_t)(4 * sa) * H + c0 + sq;
  // this lane's A row (tile row 16 wr + lane % 16) and first k (4 per lane group)
  const int lr = 16 * wr + (lane & 15);
  const int sample = mma ? idx[(lr < 32 ? slot_a : slot_b) * kBatch + (lr & 31)] : 0;
  const float* arow = data + (int64_t)sample * d.d_in + 4 * (lane >> 4);
  __bf16* my_bs = Bs + half * 2 * kStage;

  struct Regs {
    f32x4 w[4], a[4];
  };
  auto load = [&](Regs& R, int chunk) {
    const int k0 = chunk * kKc;
#pragma unroll
    for (int r = 0; r < 4; ++r) R.w[r] = *reinterpret_cast<const f32x4*>(wsrc + (int64_t)(k0 + r) * H);
    if (mma) {
#pragma unroll
      for (int u = 0; u < 4; ++u)
        R.a[u] = *reinterpret_cast<const f32x4*>(arow + k0 + 16 * u);
    }
  };
  bf16x8 fa[2], fn[2];  // A fragments (K steps 0, 1) of the current and the next chunk
  // K order within a 64-deep chunk: the MFMA sums over its 32 K slots in any
  // order, so slot (step ks, lane group g, element t) takes k = 32 ks +
  // 16 (t / 4) + 4 g + t % 4.  Then a lane's A values of one load are 4
  // consecutive k, and the four lane groups of a row read 64 contiguous bytes.
  // The staged chunk is [unit][k] in 16-byte pieces, piece 4 ks + g holding
  // that fragment's 8 k; piece c of unit u sits at position c ^ ((u / 8) % 8)
  // of its row, so that the fragment reads spread over all LDS banks.
  auto stage = [&](const Regs& R, int buf) {
    __bf16* b = my_bs + buf * kStage + 8 * ((4 * (sa >> 3) + (sa & 3)) ^ ((sq >> 3) & 7)) +
                4 * ((sa >> 2) & 1);
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const uint2 v = {pack_bf16(R.w[0][t], R.w[1][t]), pack_bf16(R.w[2][t], R.w[3][t])};
      *reinterpret_cast<uint2*>(b + (sq + t) * kLdb) = v;
    }
    if (mma) {
#pragma unroll
      for (int ks = 0; ks < 2; ++ks)
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          fn[ks][t] = (__bf16)R.a[2 * ks][t];
          fn[ks][t + 4] = (__bf16)R.a[2 * ks + 1][t];
        }
    }
  };

  f32x4 acc[4];
#pragma unroll
  for (int ct = 0; ct < 4; ++ct) acc[ct] = f32x4{0.f, 0.f, 0.f, 0.f};
  auto multiply = [&](int buf) {
    if (!mma) return;
    const __bf16* bs = my_bs + buf * kStage + (lane & 15) * kLdb;
    const int piece = lane >> 4, swz = (lane & 15) >> 3;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
      for (int ct = 0; ct < 4; ++ct) {
        const int col = 8 * ((piece + 4 * ks) ^ (swz + 2 * ct));
        const bf16x8 fb = *reinterpret_cast<const bf16x8*>(bs + 16 * ct * kLdb + col);
        acc[ct] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[ks], fb, acc[ct], 0, 0, 0);
      }
  };
  // half h takes chunks h, h+2, ...: S of them (d_in % 128 == 0, so every
  // half has the same count); chunk s of this half is 2 s + h.  Register set
  // c % kDepth holds chunk c from its load until it is staged.
  const int S = d.d_in / (2 * kKc);
  Regs R[kDepth];
#pragma unroll
  for (int c = 0; c < kDepth; ++c)
    if (c < S) load(R[c], 2 * c + half);
  stage(R[0], 0);
  fa[0] = fn[0];
  fa[1] = fn[1];
  if (kDepth < S) load(R[0], 2 * kDepth + half);
  __syncthreads();
  // step s: multiply chunk s (LDS buffer s % 2); stage chunk s+1 from its
  // register set and refill that set with chunk s+1+kDepth
  auto step = [&](int s, Regs& Rn) {
    multiply(s & 1);
    if (s + 1 < S) stage(Rn, (s + 1) & 1);
    if (s + 1 + kDepth < S) load(Rn, 2 * (s + 1 + kDepth) + half);
    __syncthreads();
    fa[0] = fn[0];
    fa[1] = fn[1];
  };
  for (int s = 0; s < S; s += kDepth) {
#pragma unroll
    for (int j = 0; j < kDepth; ++j)
      if (s + j < S) step(s + j, R[(j + 1) % kDepth]);
  }

  // half 1 hands its sums to half 0 through LDS
  float* part = reinterpret_cast<float*>(Bs);  // [64][kLdp]
  if (half == 1 && mma) {
#pragma unroll
    for (int ct = 0; ct < 4; ++ct)
#pragma unroll
      for (int t = 0; t < 4; ++t)
        part[(16 * wr + 4 * (lane >> 4) + t) * kLdp + 16 * ct + (lane & 15)] = acc[ct][t];
  }
  __syncthreads();
  if (half == 0 && mma) {
#pragma unroll
    for (int ct = 0; ct < 4; ++ct) {
      const int col = 16 * ct + (lane & 15);
      const float b = prm[d.off_b1 + c0 + col];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int r = 16 * wr + 4 * (lane >> 4) + t;
        const float z = acc[ct][t] + part[r * kLdp + col] + b;
        Z1[((int64_t)(r < 32 ? slot_a : slot_b) * kBatch + (r & 31)) * H + c0 + col] = z;
        Hs[r * kLdh + col] = bf16r(fmaxf(z, 0.0f));
      }
    }
  }
  for (int k = tid; k < 64 * C; k += 512) W2s[k] = bf16r(prm[d.off_w2 + (int64_t)c0 * C + k]);
  __syncthreads();
  for (int o = tid; o < rows * C; o += 512) {
    const int r = o / C, c = o % C;
    float s = 0.0f;
    for (int h = 0; h < 64; ++h) s += Hs[r * kLdh + h] * W2s[h * C + c];
    Zp[(int64_t)(c0 / 64) * zp_stride +
       ((int64_t)(r < 32 ? slot_a : slot_b) * kBatch + (r & 31)) * kMaxClasses + c] = s;
  }
}

// Per mini-batch (blockIdx.x) and 64 hidden units (blockIdx.y): the logits
// (shares summed in unit-block order, + b2), softmax cross-entropy and dZ2 =
// (softmax - onehot) / 32 (recomputed by every unit block: 32 x classes
// values).  Unit block 0 writes the loss and, when BACKWARD, db2 and the
// padding of G.  When BACKWARD, wave w takes the 16 units c0 + 16w .. on
// the matrix cores: dZ1 = (bf16(dZ2) bf16(W2)^T) * [Z1 > 0] (K = classes,
// zero-padded to 32), stored in bf16 as [slot][unit][row] for k_mlp_wgrad,
// db1 = its sum over the rows, and dW2 = bf16(relu(Z1))^T bf16(dZ2) (K = the
// 32 rows).
template <bool BACKWARD>
__global__ void __launch_bounds__(256)
    k_mlp_head(const float* __restrict__ X, const int32_t* __restrict__ ylab,
               const float* __restrict__ Z1, const float* __restrict__ Zp, int64_t zp_stride,
               __bf16* __restrict__ dZ1t, float* __restrict__ G, float* __restrict__ losses, Dims d,
               List L) {
  constexpr int kLdz = 64 + 1;
  __shared__ float Zs[kBatch * kMaxClasses];  // logits, then dZ2
  __shared__ float Zb[kBatch * kMaxClasses];  // bf16(dZ2), zero beyond the classes
  __shared__ float W2s[64 * kMaxClasses];     // bf16(W2) of this block's units
  __shared__ float Z1s[kBatch * kLdz];        // Z1 of this block's units
  __shared__ float row_loss[kBatch];
  __shared__ int ys[kBatch];
  const uint32_t item = L.w[blockIdx.x];
  const int slot = item_slot_a(item);
  const float* prm = X + (int64_t)item_learner(item) * d.ld;
  const int H = d.hidden, C = d.classes;
  const int blocks = H / 64;
  const int c0 = blockIdx.y * 64;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t row0 = (int64_t)slot * kBatch;

  // every load of this phase is independent of the others
  for (int o = tid; o < kBatch * C; o += 256) {
    const int r = o / C, c = o % C;
    float z = 0.0f;
    for (int q = 0; q < blocks; ++q) z += Zp[(int64_t)q * zp_stride + (row0 + r) * kMaxClasses + c];
    Zs[r * kMaxClasses + c] = z + prm[d.off_b2 + c];
  }
  if (tid < kBatch) ys[tid] = ylab[row0 + tid];
  if (BACKWARD) {
    for (int k = tid; k < 64 * C; k += 256) W2s[k] = bf16r(prm[d.off_w2 + (int64_t)c0 * C + k]);
#pragma unroll
    for (int u = 0; u < kBatch * 64 / 256; ++u) {
      const int o = tid + 256 * u, r = o >> 6, h = o & 63;
      Z1s[r * kLdz + h] = Z1[(row0 + r) * H + c0 + h];
    }
  }
  __syncthreads();
  if (tid < kBatch) {
    const int r = tid;
    const float* z = Zs + r * kMaxClasses;
    float zmax = z[0];
    for (int c = 1; c < C; ++c) zmax = fmaxf(zmax, z[c]);
    float sum = 0.0f;
    for (int c = 0; c < C; ++c) sum += expf(z[c] - zmax);
    const float lse = zmax + logf(sum);
    row_loss[r] = lse - z[ys[r]];
    if (BACKWARD)
      for (int c = 0; c < kMaxClasses; ++c) {
        const float g = c < C ? (expf(z[c] - lse) - (c == ys[r] ? 1.0f : 0.0f)) * (1.0f / kBatch) : 0.0f;
        Zs[r * kMaxClasses + c] = g;
        Zb[r * kMaxClasses + c] = bf16r(g);
      }
  }
  __syncthreads();
  float* g = G + (int64_t)slot * d.ld;
  if (blockIdx.y == 0) {
    if (tid == 0) {
      float s = 0.0f;
      for (int r = 0; r < kBatch; ++r) s += row_loss[r];
      losses[slot] = s * (1.0f / kBatch);
    }
    if (BACKWARD) {
      if (tid < C) {
        float s = 0.0f;
        for (int r = 0; r < kBatch; ++r) s += Zs[r * kMaxClasses + tid];
        g[d.off_b2 + tid] = s;
      }
      if (tid < d.P - d.off_pad) g[d.off_pad + tid] = 0.0f;
    }
  }
  if (!BACKWARD) return;
  const int hl = 16 * wave + (lane & 15);  // this lane's unit within the block
  const int kq = 8 * (lane >> 4);          // this lane's K offset in a fragment
  // dZ1 for rows 16 rt .. +15 and units 16w .. +15
  bf16x8 fw;  // B[k][h] = bf16(W2[h][k]), k = class
#pragma unroll
  for (int t = 0; t < 8; ++t) fw[t] = (__bf16)(kq + t < C ? W2s[hl * C + kq + t] : 0.0f);
  float db1 = 0.0f;
#pragma unroll
  for (int rt = 0; rt < 2; ++rt) {
    bf16x8 fz;  // A[r][k] = bf16(dZ2[r][k])
#pragma unroll
    for (int t = 0; t < 8; ++t) fz[t] = (__bf16)(kq + t < kMaxClasses ? Zb[(16 * rt + (lane & 15)) * kMaxClasses + kq + t] : 0.0f);
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fz, fw, acc, 0, 0, 0);
    // lane holds rows 16 rt + 4 (lane / 16) + t of unit hl
    const int r0 = 16 * rt + 4 * (lane >> 4);
    float v[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      v[t] = Z1s[(r0 + t) * kLdz + hl] > 0.0f ? acc[t] : 0.0f;
      db1 += v[t];
    }
    const uint2 packed = {pack_bf16(v[0], v[1]), pack_bf16(v[2], v[3])};
    *reinterpret_cast<uint2*>(dZ1t + ((int64_t)slot * H + c0 + hl) * kBatch + r0) = packed;
  }
  // db1: the four row groups of a unit sit in lanes l, l+16, l+32, l+48
  db1 += __shfl_xor(db1, 16);
  db1 += __shfl_xor(db1, 32);
  if (lane < 16) g[d.off_b1 + c0 + hl] = db1;
  // dW2[h][c] for units 16w .. +15: A[h][r] = bf16(relu(Z1[r][h])), B[r][c] = bf16(dZ2[r][c])
  {
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
        const int h = c0 + 16 * wave + 4 * (lane >> 4) + t;
        g[d.off_w2 + (int64_t)h * C + c] = acc[t];
      }
    }
  }
}

// dW1[f][h] = sum_r bf16(A[s_r][f]) bf16(dZ1[r][h]) for one mini-batch
// (blockIdx.x) and 128 features f0 .. f0+127 (blockIdx.y), every unit h.
// Computed transposed, D[h][f] = dZ1^T A: the A operand (8 rows r of one
// unit) is a 16-byte read of the [slot][unit][row] dZ1 copy, the B operand (8
// rows of one feature) comes from the sample rows staged transposed in LDS,
// and each lane's four results are consecutive units of one G row: one
// 16-byte store.  Wave w takes unit tiles w, w+4, ...; a workgroup writes
// 128 whole G rows of dW1.
__global__ void __launch_bounds__(256)
    k_mlp_wgrad(const float* __restrict__ data, const int32_t* __restrict__ idx,
                const __bf16* __restrict__ dZ1t, float* __restrict__ G, Dims d, List L) {
  constexpr int kLda = kBatch + 8;  // bf16 per transposed sample column (16-byte aligned)
  __shared__ __attribute__((aligned(16))) __bf16 At[kFeatBlock * kLda];
  const int slot = item_slot_a(L.w[blockIdx.x]);
  const int f0 = blockIdx.y * kFeatBlock;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int H = d.hidden;
  const int64_t row0 = (int64_t)slot * kBatch;
  // this wave's dZ1 fragments (unit tiles wave, wave+4, ... < H/16 <= 32),
  // loaded before the sample rows so both latencies overlap
  const __bf16* dz = dZ1t + row0 * H + 8 * (lane >> 4);  // [unit][row] of this mini-batch
  bf16x8 fa[kMaxHidden / 64];
#pragma unroll
  for (int u = 0; u < kMaxHidden / 64; ++u) {
    const int ht = wave + 4 * u;
    if (16 * ht < H) fa[u] = *reinterpret_cast<const bf16x8*>(dz + (int64_t)(16 * ht + (lane & 15)) * kBatch);
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
  float* g = G + (int64_t)slot * d.ld + (int64_t)(f0 + (lane & 15)) * H + 4 * (lane >> 4);
#pragma unroll
  for (int u = 0; u < kMaxHidden / 64; ++u) {
    const int ht = wave + 4 * u;
    if (16 * ht >= H) break;
#pragma unroll
    for (int ft = 0; ft < kFeatBlock / 16; ++ft) {
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[u], fb[ft], acc, 0, 0, 0);
      *reinterpret_cast<f32x4*>(g + (int64_t)(16 * ft) * H + 16 * ht) = acc;
    }
  }
}

// ------------------------------------------------------------------ host

nbsgd_status check_shape(const nbsgd_mlp_shape* s, Dims* d) {
  if (!s) return fail(NBSGD_E_ARG, "shape is null");
  if (s->batch != kBatch)
    return fail(NBSGD_E_UNSUPPORTED, "batch=%d: only %d is supported", s->batch, kBatch);
  if (s->d_in < kFeatBlock || s->d_in % kFeatBlock || s->hidden < 64 || s->hidden % 64 ||
      s->hidden > kMaxHidden)
    return fail(NBSGD_E_UNSUPPORTED,
                "d_in=%d must be a multiple of %d and hidden=%d a multiple of 64, at most %d",
                s->d_in, kFeatBlock, s->hidden, kMaxHidden);
  if (s->classes < 2 || s->classes > kMaxClasses)
    return fail(NBSGD_E_UNSUPPORTED, "classes=%d must be in [2, %d]", s->classes, kMaxClasses);
  d->d_in = s->d_in;
  d->hidden = s->hidden;
  d->classes = s->classes;
  d->off_b1 = (int64_t)s->d_in * s->hidden;
  d->off_w2 = d->off_b1 + s->hidden;
  d->off_b2 = d->off_w2 + (int64_t)s->hidden * s->classes;
  d->off_pad = d->off_b2 + s->classes;
  d->P = (d->off_pad + 3) & ~(int64_t)3;
  d->ld = d->P;
  return NBSGD_OK;
}

size_t up256(size_t b) { return (b + 255) & ~(size_t)255; }

// sample list, labels, Z1 [rows][hidden] fp32, hidden/64 logit-share planes
// [rows][16] fp32 and dZ1 [rows/32][hidden][32] bf16, each 256-byte aligned
size_t workspace_for(const Dims& d, int64_t rows) {
  return 2 * up256((size_t)rows * 4) + up256((size_t)rows * d.hidden * 4) +
         (size_t)(d.hidden / 64) * up256((size_t)rows * kMaxClasses * 4) +
         up256((size_t)rows * d.hidden * 2);
}

struct Workspace {
  int32_t* idx;
  int32_t* ylab;
  float* z1;
  float* zp;
  int64_t zp_stride;  // floats between logit-share planes
  __bf16* dz1t;
};

Workspace carve(void* ws, const Dims& d, int64_t rows) {
  char* p = static_cast<char*>(ws);
  Workspace w;
  w.idx = reinterpret_cast<int32_t*>(p);
  p += up256((size_t)rows * 4);
  w.ylab = reinterpret_cast<int32_t*>(p);
  p += up256((size_t)rows * 4);
  w.z1 = reinterpret_cast<float*>(p);
  p += up256((size_t)rows * d.hidden * 4);
  w.zp = reinterpret_cast<float*>(p);
  w.zp_stride = (int64_t)(up256((size_t)rows * kMaxClasses * 4) / 4);
  p += (size_t)(d.hidden / 64) * up256((size_t)rows * kMaxClasses * 4);
  w.dz1t = reinterpret_cast<__bf16*>(p);
  return w;
}

// Copies the sample indices of the mini-batches `slots` (host idx[slot*32 ..])
// to the workspace through kernel arguments, after checking every one.
nbsgd_status upload_idx(const int32_t* host, const int32_t* slots, int n_slots, int64_t n_samples,
                        const int32_t* labels, const Dims& d, const Workspace& w, hipStream_t s) {
  for (int k = 0; k < n_slots; ++k)
    for (int r = 0; r < kBatch; ++r) {
      const int64_t pos = (int64_t)slots[k] * kBatch + r;
      if (host[pos] < 0 || host[pos] >= n_samples)
        return fail(NBSGD_E_ARG, "sample index %d at position %lld is outside [0, %lld)", host[pos],
                    (long long)pos, (long long)n_samples);
    }
  const int wide = n_samples > 65536 ? 1 : 0;
  const int per = wide ? kUpSlots / 2 : kUpSlots;
  for (int k0 = 0; k0 < n_slots; k0 += per) {
    IdxChunk c;
    memset(&c, 0, sizeof(c));
    c.n_slots = std::min(per, n_slots - k0);
    c.wide = wide;
    for (int k = 0; k < c.n_slots; ++k) {
      c.slot[k >> 1] |= (uint32_t)slots[k0 + k] << (16 * (k & 1));
      const int32_t* src = host + (int64_t)slots[k0 + k] * kBatch;
      for (int r = 0; r < kBatch; ++r) {
        const int t = k * kBatch + r;
        if (wide) c.v[t] = (uint32_t)src[r];
        else c.v[t >> 1] |= (uint32_t)src[r] << (16 * (t & 1));
      }
    }
    hipLaunchKernelGGL(k_put_idx, dim3((c.n_slots * kBatch + 255) / 256), dim3(256), 0, s, w.idx,
                       w.ylab, labels, d.classes, c);
  }
  return NBSGD_OK;
}

nbsgd_status launch_err(const char* what) {
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(NBSGD_E_HIP, "%s launch failed: %s", what, hipGetErrorString(e));
  return NBSGD_OK;
}

uint32_t item(int learner, int slot_a, int slot_b) {
  return ((uint32_t)learner << 24) | ((uint32_t)slot_a << 12) | (uint32_t)(slot_b + 1);
}

// Launches the three kernels over mini-batches `mb` (learner, slot), sorted
// by learner, of one group (at most kMaxList): forward tiles pair
// consecutive mini-batches of the same learner.
template <bool BACKWARD>
void launch_group(const std::pair<int, int>* mb, int count, const float* X, const float* data,
                  const Workspace& w, float* G, float* losses, const Dims& d, hipStream_t st) {
  const int nb = d.hidden / 64;
  List tiles, items;
  FwdMap M;
  tiles.count = items.count = 0;
  M.n = 0;
  int total = 0;
  for (int k = 0; k < count; ++k) {
    if (k == 0 || mb[k].first != mb[k - 1].first) {  // a new learner
      if (M.n > 0) total += nb * (tiles.count - M.first[M.n - 1]);
      M.off[M.n] = total;
      M.first[M.n] = tiles.count;
      ++M.n;
    }
    items.w[items.count++] = item(mb[k].first, mb[k].second, -1);
    if (k + 1 < count && mb[k + 1].first == mb[k].first) {
      tiles.w[tiles.count++] = item(mb[k].first, mb[k].second, mb[k + 1].second);
      ++k;
      items.w[items.count++] = item(mb[k].first, mb[k].second, -1);
    } else {
      tiles.w[tiles.count++] = item(mb[k].first, mb[k].second, -1);
    }
  }
  total += nb * (tiles.count - M.first[M.n - 1]);
  M.off[M.n] = total;
  M.first[M.n] = tiles.count;
  for (int x = 0; x <= 8; ++x) M.xcd_start[x] = (int32_t)((int64_t)x * total / 8);
  const int per_xcd = (total + 7) / 8;
  hipLaunchKernelGGL(k_mlp_fwd, dim3(8 * per_xcd), dim3(512), 0, st, X, data, w.idx, w.z1, w.zp,
                     w.zp_stride, d, M, tiles);
  hipLaunchKernelGGL(k_mlp_head<BACKWARD>, dim3(items.count, BACKWARD ? nb : 1), dim3(256), 0, st, X,
                     w.ylab, w.z1, w.zp, w.zp_stride, w.dz1t, G, losses, d, items);
  if (BACKWARD)
    hipLaunchKernelGGL(k_mlp_wgrad, dim3(items.count, d.d_in / kFeatBlock), dim3(256), 0, st, data,
                       w.idx, w.dz1t, G, d, items);
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

namespace {

nbsgd_status mlp_grad_impl(const float* X, int64_t ld, int32_t n, int32_t m,
                           const nbsgd_mlp_shape* s, const float* data, const int32_t* labels,
                           int64_t n_samples, const int32_t* idx, const uint8_t* mask, float* G,
                           float* losses, void* workspace, size_t workspace_bytes, void* stream) {
  if (nbsgd_status st = check_nm(n, m)) return st;
  Dims d;
  if (nbsgd_status st = check_shape(s, &d)) return st;
  if (ld == 0) ld = d.P;
  if (ld < d.P || ld % 4)
    return fail(NBSGD_E_SHAPE, "row stride %lld must be a multiple of 4 and at least P=%lld",
                (long long)ld, (long long)d.P);
  d.ld = ld;
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
  std::vector<int32_t> finished;
  for (int32_t k = 0; k < n * m; ++k)
    if (mask[k]) finished.push_back(k);
  if (nbsgd_status r = upload_idx(idx, finished.data(), (int)finished.size(), n_samples, labels, d, w, st))
    return r;
  std::pair<int, int> mb[kMaxList];
  int count = 0;
  for (int32_t k : finished) {
    mb[count++] = {k / m, k};
    if (count == kMaxList) {
      launch_group<true>(mb, count, X, data, w, G, losses, d, st);
      count = 0;
    }
  }
  if (count) launch_group<true>(mb, count, X, data, w, G, losses, d, st);
  return launch_err("nbsgd_mlp_grad");
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
  if (nbsgd_status r = upload_idx(idx, slots, count / kBatch, n_samples, labels, d, w, st)) return r;
  launch_group<false>(mb, count / kBatch, params, data, w, nullptr, losses, d, st);
  return launch_err("nbsgd_mlp_loss");
}
