/*
 * nbsgd.h - C ABI of libnbsgd, the MI355X (gfx950) hot path of Non-blocking SGD
 * (He & Dube, "Accelerating Parallel Stochastic Gradient Descent via
 * Non-blocking Mini-batches", arXiv 2211.00889).
 *
 * n learners are simulated as parameter replicas resident in one GPU's HBM.
 * One iteration (Alg. 2) is:
 *   1. every learner processes its mini-batches in order until the fastest
 *      learner, having finished all m, broadcasts the terminal signal; the
 *      unfinished mini-batches are abandoned            -> nbsgd_sample_mask
 *   2. each learner averages the gradients of its finished mini-batches
 *                                                        -> nbsgd_accumulate
 *   3. models are averaged through a doubly stochastic mixing matrix W
 *      (ring all-reduce, D-PSGD ring gossip or MATCHA)   -> nbsgd_mix
 *   4. each learner takes one local step with learning rate lr * c_i / m,
 *      here with heavy-ball momentum                     -> nbsgd_update
 * nbsgd_step does 2-4 in one pass over HBM.
 *
 * Notation: n learners (the paper's P), m mini-batches per learner per
 * iteration (the paper's N), P parameters per replica (the paper's d),
 * c_i finished mini-batches of learner i (the paper's n_{k,i}).
 *
 * Conventions for every call:
 *   - returns nbsgd_status; NBSGD_OK is 0.  On error nothing is enqueued and
 *     nbsgd_last_error() (thread-local) describes the first failed check.
 *   - device buffers are fp32, contiguous, row-major, caller-owned (typically
 *     torch.empty(..., device="cuda")); the library never retains or frees a
 *     pointer.  Base pointers must be 16-byte aligned (NBSGD_E_ALIGN).
 *   - host arrays (mask, counts, W) are read completely before the call
 *     returns; the caller may reuse them at once.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *     Kernels are enqueued asynchronously; device faults surface at the
 *     caller's next synchronisation.  No hot call allocates or synchronises.
 *   - limits: 1 <= n <= NBSGD_MAX_LEARNERS, 1 <= m <= NBSGD_MAX_MINIBATCHES
 *     (NBSGD_E_UNSUPPORTED beyond); P >= 0, P == 0 is a valid empty call.
 *   - all functions are reentrant; calls on one stream execute in order.
 */
#ifndef NBSGD_H
#define NBSGD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define NBSGD_MAX_LEARNERS 16
#define NBSGD_MAX_MINIBATCHES 64

typedef enum {
  NBSGD_OK = 0,
  NBSGD_E_ARG = 1,         /* null pointer, bad enum, overlapping buffers */
  NBSGD_E_SHAPE = 2,       /* negative or inconsistent sizes */
  NBSGD_E_ALIGN = 3,       /* device base pointer not 16-byte aligned */
  NBSGD_E_MASK = 4,        /* a learner with no finished mini-batch */
  NBSGD_E_W = 5,           /* W not finite, negative, or not doubly stochastic */
  NBSGD_E_HIP = 6,         /* a HIP runtime call or kernel launch failed */
  NBSGD_E_UNSUPPORTED = 7  /* n or m beyond the compiled limits */
} nbsgd_status;

/* Order of the averaging and the local step.  MIX_THEN_STEP averages the
 * pre-step models and subtracts each learner's own step (Alg. 2, averaging
 * then update).  STEP_THEN_MIX steps first and averages the stepped models
 * (Eq. 4-5 ring all-reduce, Eq. 6 D-PSGD, Alg. 3). */
typedef enum { NBSGD_MIX_THEN_STEP = 0, NBSGD_STEP_THEN_MIX = 1 } nbsgd_order;

/* Per-mini-batch time model: t = s_i * (base + D) with the learner's
 * slow-down s_i:
 *   slow_learner >= 0: s_i = slow_factor for that learner, 1 for the others;
 *   slow_learner == NBSGD_SLOW_NONE (-1): s_i = 1;
 *   slow_learner == NBSGD_SLOW_RANDOM (-2): the paper's heterogeneity model
 *     (Sec. 6.1: the slowed nodes and the rate of slow-down change every
 *     iteration, the slowest node taking up to twice as long): at each
 *     iteration every learner is slowed with probability slow_prob, by a
 *     factor 1 + (slow_factor - 1) * u, u uniform in (0, 1) (words 0 and 1
 *     of Philox4x64-10 at counter (step, i, 0, 0) under key (seed, 5): slowed
 *     iff u0 < slow_prob, factor from u1, both mapped as below).
 *   CONST: D = 0
 *   EXP:   D ~ Exp(rate = param), mean 1/param (App. A, Remark 1)
 *   LOMAX: D = Pareto type II with shape param, so base 1 + D is Pareto with
 *          scale 1 (heavy-tailed stragglers)                                  */
typedef enum { NBSGD_DELAY_CONST = 0, NBSGD_DELAY_EXP = 1, NBSGD_DELAY_LOMAX = 2 } nbsgd_delay_kind;

#define NBSGD_SLOW_NONE (-1)
#define NBSGD_SLOW_RANDOM (-2)

typedef struct {
  int32_t kind;        /* nbsgd_delay_kind */
  double base;         /* >= 0 */
  double param;        /* EXP: rate > 0; LOMAX: shape > 0 (finite); CONST: ignored */
  int32_t slow_learner;
  double slow_factor;  /* finite, > 0; >= 1 for NBSGD_SLOW_RANDOM */
  double slow_prob;    /* NBSGD_SLOW_RANDOM only: in [0, 1] */
} nbsgd_delay;

/* ---------------------------------------------------------------- schedule
 * Simulated terminal signal of one iteration (Alg. 2 mini-batch loop; Lemma 1).
 * Mini-batch j of learner i at iteration `step` takes t[i][j] (delay model
 * above; the uniform variate is Philox4x64-10 word 0 at counter
 * (step, i, j, 0) under key (seed, 1), mapped to ((w >> 12) + 0.5) * 2^-52).
 * With C[i][j] the running sum of t[i][0..j] (fp64, j ascending), the signal
 * comes at T = min_i C[i][m-1]; learner i finished c_i = max(1, #{j :
 * C[i][j] <= T}) mini-batches, its first c_i.
 * Outputs (host, caller-owned):
 *   mask   uint8[n*m], row-major: mask[i*m+j] = 1 iff j < c_i
 *   counts int32[n]:   c_i
 *   times  double[n*m] (nullable): t[i][j]
 *   timing double[3]   (nullable): {T, T_sync = max_i C[i][m-1] (the blocking
 *          iteration time), T_step = max(T, max_i C[i][c_i-1])}
 * Errors: NBSGD_E_ARG (null mask/counts/d, bad kind or non-positive param,
 *         slow_learner below -2 or at least n, a slow-down outside its range),
 *         NBSGD_E_SHAPE, NBSGD_E_UNSUPPORTED.                                  */
nbsgd_status nbsgd_sample_mask(uint64_t seed, uint64_t step, int32_t n, int32_t m,
                               const nbsgd_delay *d, uint8_t *mask, int32_t *counts,
                               double *times, double *timing);

/* -------------------------------------------------- Sec. 4.3 accounting
 * Throughput accounting of one iteration (Thm 3-5, Cor. 1) from its
 * per-mini-batch times (the `times` output of nbsgd_sample_mask), in units of
 * mini-batches: a learner's batch B is its m mini-batches.  Learner i's batch
 * time is X_i = sum_j times[i*m+j] (summed in mini-batch order); X_{1:P} <=
 * ... <= X_{P:P} are the X_i sorted, and Y = sum_k 1 / X_{k:P}, summed from
 * the fastest learner.
 *   x_first          X_{1:P}: the non-blocking iteration time (the terminal
 *                    signal, T of nbsgd_sample_mask)
 *   x_last           X_{P:P}: the blocking iteration time (T_sync)
 *   y                Y
 *   throughput       Thm 3: B * Y, non-blocking mini-batches per time unit
 *   throughput_sync  Thm 4: P * B / X_{P:P}, the blocking baseline's
 *   data             Cor. 1: B * Y * X_{1:P}, the fractional number of
 *                    mini-batches one non-blocking iteration trains when
 *                    every learner runs at a constant speed within it
 *   ratio            Thm 5: Y * X_{P:P} / P, non-blocking over blocking
 *                    throughput (>= 1)
 * times  host double [n*m], finite and >= 0, every learner's sum > 0.
 * Errors: NBSGD_E_ARG (null pointer, a negative or non-finite time, a zero
 *         batch time), NBSGD_E_SHAPE, NBSGD_E_UNSUPPORTED.                    */
typedef struct {
  double x_first, x_last, y, throughput, throughput_sync, data, ratio;
} nbsgd_accounting;
nbsgd_status nbsgd_iteration_accounting(const double *times, int32_t n, int32_t m,
                                        nbsgd_accounting *out);

/* ------------------------------------------------------------- accumulate
 * Accumulated gradient of the finished mini-batches (Alg. 2 mini-batch loop;
 * Sec. 3.2, gradient bullet), normalised by the finished count:
 *   Gbar[i][:] = (1 / c_i) * sum_{j : mask[i*m+j] != 0} G[i][j][:]
 * G     device fp32 [n][m][P] (only finished rows are read)
 * mask  host uint8 [n*m], any pattern; c_i = number of nonzero entries >= 1
 * Gbar  device fp32 [n][P], written; must not overlap G
 * Errors: NBSGD_E_ARG, NBSGD_E_SHAPE, NBSGD_E_ALIGN, NBSGD_E_MASK,
 *         NBSGD_E_UNSUPPORTED, NBSGD_E_HIP.                                    */
nbsgd_status nbsgd_accumulate(const float *G, const uint8_t *mask, int32_t n, int32_t m,
                              int64_t P, float *Gbar, void *stream);

/* -------------------------------------------------------------------- mix
 * Neighbourhood averaging (Alg. 2 averaging step; Eq. 6):
 *   Y[i][:] = sum_p W[i*n+p] * X[p][:]
 * X, Y  device fp32 [n][P]; Y == X (in place) is allowed, partial overlap is
 *       not (NBSGD_E_ARG)
 * W     host fp32 [n*n], row-major; entries finite and >= 0, every row and
 *       column sum within 1e-5 of 1 (NBSGD_E_W).  Zero entries are skipped; a
 *       W whose entries are all equal (ring all-reduce, J/n) takes a path that
 *       sums once and scales, so every row of Y is bitwise identical.
 * Errors: NBSGD_E_ARG, NBSGD_E_SHAPE, NBSGD_E_ALIGN, NBSGD_E_W,
 *         NBSGD_E_UNSUPPORTED, NBSGD_E_HIP.                                    */
nbsgd_status nbsgd_mix(const float *X, const float *W, int32_t n, int64_t P, float *Y,
                       void *stream);

/* ----------------------------------------------------------------- update
 * Local step with the finished-fraction learning rate (Sec. 3.2, learning-rate
 * and update bullets) and heavy-ball momentum:
 *   eta_i = lr * counts[i] / m   (fp64, rounded once to fp32)
 *   V[i] = momentum * V[i] + Gbar[i];   X[i] = X[i] - eta_i * V[i]
 * X, V  device fp32 [n][P], updated in place
 * Gbar  device fp32 [n][P] (from nbsgd_accumulate)
 * counts host int32 [n], 1 <= counts[i] <= m
 * Errors: NBSGD_E_ARG, NBSGD_E_SHAPE, NBSGD_E_ALIGN, NBSGD_E_MASK (a count
 *         outside [1, m]), NBSGD_E_UNSUPPORTED, NBSGD_E_HIP.                  */
nbsgd_status nbsgd_update(float *X, float *V, const float *Gbar, const int32_t *counts, int32_t n,
                          int32_t m, int64_t P, float lr, float momentum, void *stream);

/* ------------------------------------------------------------------- step
 * One whole Non-blocking iteration after the schedule (Alg. 2), fused so X, V
 * and the finished rows of G each cross HBM once:
 *   g_i   = (1/c_i) sum_{finished j} G[i][j]     eta_i = lr * c_i / m
 *   V[i]  = momentum * V[i] + g_i
 *   MIX_THEN_STEP: X[i] = sum_p W[i*n+p] X[p] - eta_i V[i]
 *   STEP_THEN_MIX: X[i] = sum_p W[i*n+p] (X[p] - eta_p V[p])
 * Equal, up to fp32 rounding, to accumulate + mix + update (MIX_THEN_STEP) or
 * accumulate + update + mix (STEP_THEN_MIX).  Non-blocking synchronous
 * centralized SGD (Alg. 3, with the 1/n of Eq. 2) is STEP_THEN_MIX with the
 * uniform W on replicas that all hold the server model: every row of X then
 * becomes x_ps - (1/n) sum_i eta_i V[i].
 * X, V  device fp32 [n][P], updated in place; G device fp32 [n][m][P], must
 *       not overlap X or V; X and V must not overlap.
 * mask, W as above; order is an nbsgd_order.
 * Errors: NBSGD_E_ARG, NBSGD_E_SHAPE, NBSGD_E_ALIGN, NBSGD_E_MASK, NBSGD_E_W,
 *         NBSGD_E_UNSUPPORTED, NBSGD_E_HIP.                                    */
nbsgd_status nbsgd_step(float *X, float *V, const float *G, const uint8_t *mask, const float *W,
                        int32_t n, int32_t m, int64_t P, float lr, float momentum, int32_t order,
                        void *stream);

/* nbsgd_step on rows `ld` floats apart: row i of X and V starts at X + i*ld,
 * V + i*ld, and row (i, j) of G at G + (i*m + j)*ld; only the first P floats
 * of a row are read or written (the rest of each row is never touched).
 * ld >= P (NBSGD_E_SHAPE).  The vector width is the largest of 4, 2, 1
 * dividing both P and ld.  nbsgd_step is this call with ld = P.
 * Errors: as nbsgd_step.                                                    */
nbsgd_status nbsgd_step_strided(float *X, float *V, const float *G, int64_t ld,
                                const uint8_t *mask, const float *W, int32_t n, int32_t m,
                                int64_t P, float lr, float momentum, int32_t order, void *stream);

/* Non-blocking synchronous centralized SGD (Alg. 3; the 1/n of Eq. 2
 * restored): one server model x, each learner's momentum buffer and
 * accumulated gradient (its finished mini-batches, evaluated at the server
 * model by the caller), in one pass:
 *   g_i = (1/c_i) sum_{finished j} G[i][j]      eta_i = lr * c_i / m
 *   V[i] = momentum * V[i] + g_i
 *   x    = x - (1/n) sum_i eta_i V[i]   (1/n in fp32, summed in learner order)
 * x     device fp32 [P] (the server model), updated in place
 * V, G  device fp32 rows `ld` floats apart as in nbsgd_step_strided:
 *       V [n][ld] updated in place, G [n][m][ld] read (finished rows only)
 * mask  host uint8 [n*m] as in nbsgd_step.  x, V and G must not overlap.
 * HBM traffic: 4 * P * (sum_i c_i + 2n + 2) bytes, against 4 * P *
 * (sum_i c_i + 4n) for the same update on n replicas of x with nbsgd_step.
 * Errors: as nbsgd_step_strided.                                            */
nbsgd_status nbsgd_step_server(float *x, float *V, const float *G, int64_t ld, const uint8_t *mask,
                               int32_t n, int32_t m, int64_t P, float lr, float momentum,
                               void *stream);

/* Row stride (in floats) to allocate X, V and G with for nbsgd_step_strided:
 *   P <= 2^20:          P (no padding);
 *   2^20 < P <= 2^22:   the next power of two, 2^21 or 2^22;
 *   P > 2^22:           k * 2^22 with k = ceil(P / 2^22), or k + 1 when k is
 *                       a power of two, so every row starts on a 16 MiB
 *                       boundary without a power-of-two stride.
 * Measured on MI355X for the fused step: the HBM throughput depends on where
 * the rows start relative to each other (the DRAM address mapping).  Above
 * 2^22 this stride raised the sustained rate of the 11.2M-, 23.5M- and
 * 138M-parameter workloads by 3-6% (k = 3, 6, 33), whereas a power-of-two
 * stride lowered it by up to 8%; between 2^20 and 2^22 the power-of-two
 * stride was the best or close to the best of the strides tried, 0-15% above
 * unpadded rows.  The padding costs memory (up to twice the rows' size in the
 * middle band), never traffic.
 * Errors: NBSGD_E_ARG (null ld), NBSGD_E_SHAPE (P < 0).                    */
nbsgd_status nbsgd_row_stride(int64_t P, int64_t *ld);

/* ------------------------------------------------------- mixing matrices
 * Host builders, W fp32 [n*n] row-major, caller-owned.
 * nbsgd_w_allreduce: every entry 1/n (ring all-reduce averages all replicas,
 *   Eq. 4-5).
 * nbsgd_w_ring: D-PSGD on a ring (Eq. 6): W[i][i] = W[i][i+-1 mod n] = 1/3;
 *   n = 2 gives all entries 1/2, n = 1 gives [1].
 * Errors: NBSGD_E_ARG (null W), NBSGD_E_SHAPE, NBSGD_E_UNSUPPORTED.          */
nbsgd_status nbsgd_w_allreduce(int32_t n, float *W);
nbsgd_status nbsgd_w_ring(int32_t n, float *W);

/* MATCHA with a communication budget (Sec. 6.1): a random `degree`-regular
 * simple connected base graph on n nodes (pairing model; half-edge shuffle by
 * Fisher-Yates from the top with Philox4x64-10 word 0 at counter
 * (attempt, position, 0, 0) under key (seed, 2) mapped to [0, t] by
 * floor(w * (t+1) / 2^64); rejected and redrawn on a loop, a repeated edge or
 * a disconnected graph), split into matchings by greedy edge colouring in
 * lexicographic edge order.  At iteration `step` matching q is active iff
 * u < p_q, u = ((w >> 12) + 0.5) * 2^-52 from Philox word 0 at counter
 * (step, q, 0, 0) under key (seed, 3), and W = I - alpha * sum_{active q} L_q,
 * L_q the Laplacian of matching q.  By default every p_q = 1/2 (budget 0.5)
 * and alpha = 1 / (degree + 1).
 * nbsgd_matcha_create: builds the graph; *out is owned by the caller and
 *   released with nbsgd_matcha_destroy.  Errors: NBSGD_E_ARG, NBSGD_E_SHAPE
 *   (no such regular graph: n < 2, degree outside [1, n), n * degree odd,
 *   degree 1 with n > 2; or none drawn in 100,000 attempts: a pairing is
 *   simple with probability about exp(-(degree^2 - 1) / 4), so degrees of 7
 *   and more, and graphs close to complete, usually end here),
 *   NBSGD_E_UNSUPPORTED.
 * nbsgd_matcha_w: W of iteration `step`; n_active (nullable) receives the
 *   number of active matchings.
 * nbsgd_matcha_matchings: edges_uvq int32[3*E] as (u, v, matching) with u < v
 *   in lexicographic order (nullable to query sizes), *E edges, *M matchings.
 * nbsgd_matcha_set / nbsgd_matcha_get: the activation probabilities p[M] (each
 *   in [0, 1]) and alpha (in (0, 1/degree], so W stays non-negative).
 * nbsgd_matcha_optimize: MATCHA's own choice under budget b in (0, 1]: p
 *   maximising the algebraic connectivity lambda_2(sum_q p_q L_q) subject to
 *   0 <= p_q <= 1 and sum_q p_q <= b * M (projected supergradient ascent,
 *   `iterations` steps, the best iterate kept), then alpha minimising the
 *   spectral norm of E[W^T W] - J/n = I - J/n - 2 alpha Lbar
 *   + alpha^2 (Lbar^2 + 2 sum_q p_q (1 - p_q) L_q) over (0, 1/degree]
 *   (grid, then golden section).  lambda2 and spectral (nullable) receive the
 *   attained values.  Host only, O(iterations * n^3).                        */
typedef struct nbsgd_matcha nbsgd_matcha;
nbsgd_status nbsgd_matcha_create(uint64_t seed, int32_t n, int32_t degree, nbsgd_matcha **out);
nbsgd_status nbsgd_matcha_w(const nbsgd_matcha *g, uint64_t step, float *W, int32_t *n_active);
nbsgd_status nbsgd_matcha_matchings(const nbsgd_matcha *g, int32_t *edges_uvq, int32_t *E,
                                    int32_t *M);
nbsgd_status nbsgd_matcha_set(nbsgd_matcha *g, const double *probs, double alpha);
nbsgd_status nbsgd_matcha_get(const nbsgd_matcha *g, double *probs, double *alpha);
nbsgd_status nbsgd_matcha_optimize(nbsgd_matcha *g, double budget, int32_t iterations,
                                   double *lambda2, double *spectral);
void nbsgd_matcha_destroy(nbsgd_matcha *g);

/* -------------------------------------------------- end-to-end MLP workload
 * Learners train a two-layer perceptron, d_in -> hidden (ReLU) -> classes with
 * softmax cross-entropy, on a data set split into n equal shards (Alg. 1/2
 * initialisation; Eq. 1 with the per-sample cross-entropy as l).
 * Flat parameter layout of one replica row: W1[d_in][hidden] row-major,
 * b1[hidden], W2[hidden][classes], b2[classes], then zeros up to a multiple
 * of 4 floats (so that every row of X, V and G starts 16-byte aligned and the
 * fused step streams it in 16-byte vectors).
 * Supported shapes: batch == 32, d_in a multiple of 128, hidden a multiple of 64,
 * hidden <= 512, 2 <= classes <= 16 (NBSGD_E_UNSUPPORTED otherwise).        */
typedef struct {
  int32_t d_in, hidden, classes, batch;
} nbsgd_mlp_shape;

/* Parameters per replica: d_in*hidden + hidden + hidden*classes + classes,
 * rounded up to a multiple of 4 (the padding). */
nbsgd_status nbsgd_mlp_param_count(const nbsgd_mlp_shape *s, int64_t *P);

/* Device workspace, in bytes, for calls that process up to `rows` sample rows:
 * n*m*batch for nbsgd_mlp_grad, `count` for nbsgd_mlp_loss.  The caller
 * allocates it once (16-byte aligned) and may reuse it for every call on the
 * same stream; calls that overlap on different streams need their own.      */
nbsgd_status nbsgd_mlp_workspace_bytes(const nbsgd_mlp_shape *s, int64_t rows, size_t *bytes);

/* Local shuffling: each learner reshuffles its own shard at every epoch
 * boundary (Alg. 1/2 initialisation; Sec. 3.2 shuffling bullet).  Learner i owns samples
 * [shard*i, shard*(i+1)).  Local epoch e permutes its shard by Fisher-Yates
 * from the top (position t swaps with floor(w*(t+1)/2^64), w = Philox4x64-10
 * word 0 at counter (e, i, t, 0) under key (seed, 4)); iteration `step` is
 * window step mod (shard / (m*b)) of epoch step div (shard / (m*b)), and
 * mini-batch j is the j-th run of b samples of that window.  Windows are
 * consumed whether or not their mini-batches finish.  The permutations of
 * the last epoch asked for are kept per calling thread, so the iterations of
 * an epoch after the first cost O(n*m*b).
 * idx: host int32 [n][m][b], global sample indices (caller-owned).
 * Errors: NBSGD_E_ARG (null idx), NBSGD_E_SHAPE (shard < m*b, b < 1),
 *         NBSGD_E_UNSUPPORTED.                                              */
nbsgd_status nbsgd_minibatch_indices(uint64_t seed, uint64_t step, int32_t n, int32_t m, int32_t b,
                                     int32_t shard, int32_t *idx);

/* Per-mini-batch gradients (Alg. 2 mini-batch loop, gradient line; Sec. 3.2,
 * gradient bullet) of every finished mini-batch, each at its
 * learner's replica:
 *   G[i][j][:] = gradient of the mean cross-entropy of the 32 samples
 *                idx[i][j][:] at parameters X[i], for mask[i*m+j] != 0;
 *   losses[i*m+j] = that mean loss.
 * The padding entries of a finished row are set to 0.  Unfinished rows of G
 * and entries of losses are left untouched.  Every GEMM
 * input (the samples, W1, bf16(ReLU(Z1)), W2, dZ2, dZ1) is rounded to bf16
 * (nearest even) and multiplied on the matrix cores with fp32 accumulation;
 * bias, ReLU, softmax and cross-entropy are fp32.
 * X      device fp32 [n][P] (P from nbsgd_mlp_param_count)
 * data   device fp32 [n_samples][d_in]; labels device int32 [n_samples] in
 *        [0, classes) (values outside are clamped into range)
 * idx    host int32 [n*m*batch]; the entries of finished mini-batches must be
 *        in [0, n_samples) (NBSGD_E_ARG, checked before any launch); read
 *        before the call returns (copied through kernel arguments)
 * mask   host uint8 [n*m]
 * G      device fp32 [n][m][P]; losses device fp32 [n*m]
 * workspace  device, >= nbsgd_mlp_workspace_bytes(s, n*m*batch)
 * Errors: NBSGD_E_ARG, NBSGD_E_SHAPE, NBSGD_E_ALIGN, NBSGD_E_UNSUPPORTED,
 *         NBSGD_E_HIP.                                                      */
nbsgd_status nbsgd_mlp_grad(const float *X, int32_t n, int32_t m, const nbsgd_mlp_shape *s,
                            const float *data, const int32_t *labels, int64_t n_samples,
                            const int32_t *idx, const uint8_t *mask, float *G, float *losses,
                            void *workspace, size_t workspace_bytes, void *stream);

/* nbsgd_mlp_grad on rows `ld` floats apart, the layout of nbsgd_step_strided:
 * replica i is read from X + i*ld and mini-batch (i, j) written to
 * G + (i*m + j)*ld; only the first P floats of a row are read or written.
 * X needs (n-1)*ld + P floats and G (n*m-1)*ld + P.  ld must be a multiple
 * of 4 and >= P (NBSGD_E_SHAPE).  nbsgd_mlp_grad is this call with ld = P.
 * Errors: as nbsgd_mlp_grad.                                                */
nbsgd_status nbsgd_mlp_grad_strided(const float *X, int64_t ld, int32_t n, int32_t m,
                                    const nbsgd_mlp_shape *s, const float *data,
                                    const int32_t *labels, int64_t n_samples, const int32_t *idx,
                                    const uint8_t *mask, float *G, float *losses, void *workspace,
                                    size_t workspace_bytes, void *stream);

/* Allocation-free nbsgd_mlp_grad_strided, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc): the same kernels and results, bit for bit, with the
 * workspace taken from a static device buffer of NBSGD_MLP_SCRATCH_BYTES
 * (32 MiB) that every GPU the library is loaded on holds until the process
 * ends.  Nothing is allocated or freed; the buffer's device address is looked
 * up once per device (hipGetSymbolAddress, with that device current).
 * The finished mini-batches' workspace, min(finished, 896) * batch rows of
 * nbsgd_mlp_workspace_bytes, must fit the buffer (NBSGD_E_UNSUPPORTED
 * otherwise, before anything is enqueued): up to 113 finished mini-batches
 * of a 512-unit hidden layer, e.g. every mini-batch of n = 8, m = 8 (64).
 * The kernels write every byte of the buffer they later read, so nothing is
 * cleared between calls.  All calls on one GPU share its buffer: calls that
 * overlap on that GPU (other streams, other host threads) race; calls on one
 * stream run in order.  `stream` must belong to the current device
 * (NBSGD_E_ARG).  Arguments and layout as nbsgd_mlp_grad_strided.
 * Errors: as nbsgd_mlp_grad_strided, and NBSGD_E_UNSUPPORTED (too many
 * finished mini-batches for the buffer, or a device index above 63).        */
#define NBSGD_MLP_SCRATCH_BYTES (32u * 1024u * 1024u)
nbsgd_status nbsgd_mlp_grad_noalloc(const float *X, int64_t ld, int32_t n, int32_t m,
                                    const nbsgd_mlp_shape *s, const float *data,
                                    const int32_t *labels, int64_t n_samples, const int32_t *idx,
                                    const uint8_t *mask, float *G, float *losses, void *stream);

/* Mean cross-entropy of one parameter vector on `count` samples, in batches
 * of 32: losses[k] = mean loss of samples idx[32k .. 32k+31] (same precision
 * as nbsgd_mlp_grad's forward pass).  Used to evaluate the average of the
 * replicas, the method's output (Alg. 1/2 output line).
 * params device fp32 [P]; idx host int32 [count], count a multiple of 32 and
 * at most 16384; losses device fp32 [count / 32].
 * workspace  device, >= nbsgd_mlp_workspace_bytes(s, count)
 * Errors: as nbsgd_mlp_grad.                                                */
nbsgd_status nbsgd_mlp_loss(const float *params, const nbsgd_mlp_shape *s, const float *data,
                            const int32_t *labels, int64_t n_samples, const int32_t *idx,
                            int32_t count, float *losses, void *workspace, size_t workspace_bytes,
                            void *stream);

/* ---------------------------------------------------------------- errors
 * Text of the last failed check or HIP error on the calling thread ("" if
 * none).  The pointer stays valid until the next nbsgd call on the thread. */
const char *nbsgd_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* NBSGD_H */
