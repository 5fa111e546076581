/*
 * acsc.h — C ABI of the MI355X (gfx950) masking compressor and spectral
 * corrector: the hot path of one pipeline stage of the fast compressed
 * training circuit of "Communication-Efficient LLM Adaptation over
 * Decentralized GPU Meshes".
 *
 * Conventions for every entry point:
 *   - Pointers named as device buffers must be device memory of the current
 *     HIP device; the caller owns every buffer.  The library allocates no
 *     device memory and keeps no pointer after a call returns.
 *   - Work is enqueued asynchronously on `stream` (NULL = the null stream).
 *     Buffers must stay alive, and outputs unread, until the stream has
 *     reached the enqueued work.  One workspace must not serve two calls
 *     that may run concurrently.
 *   - Matrices are row-major; `ld_*` is the row stride in elements.
 *   - Every call returns ACSC_OK (0) or a negative error code, and
 *     acsc_last_error() then describes the failure (per thread).  All argument
 *     checks happen on the host before anything is enqueued, so a failed call
 *     has no side effect.  No exception or abort crosses this boundary.
 *   - bf16 data is passed as its 16-bit patterns (uint16_t storage).
 */
#ifndef ACSC_H
#define ACSC_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum acsc_dtype { ACSC_F32 = 0, ACSC_BF16 = 1 } acsc_dtype;

#define ACSC_OK 0
#define ACSC_EINVAL (-1)  /* null pointer, bad shape, K or r out of range   */
#define ACSC_EDTYPE (-2)  /* unknown dtype                                  */
#define ACSC_EALIGN (-3)  /* pointer or stride not aligned as required      */
#define ACSC_EHIP (-4)    /* HIP launch or runtime failure                  */
#define ACSC_ENOSPC (-5)  /* workspace too small                            */
#define ACSC_ENOCONV (-6) /* sc_build_status: a build did not converge, its
                             two phases did not meet on its workspace, or
                             its fused EMA pass gave up a wait              */

/* Text of the last error raised on the calling thread ("" if none). */
const char *acsc_last_error(void);

/* Library ABI version (increments on any signature change). */
int acsc_version(void);

/* Diagnostics, not part of the hot path.  acsc_stats_enable(1) resets the
 * counters and starts timing: every kernel the library enqueues from then on
 * is bracketed by a pair of HIP events recorded on its own stream, and its
 * duration is added to the total of its kernel name.  acsc_stats_enable(0)
 * stops timing.  acsc_stats_read waits for the recorded events, then returns
 * the name (NUL-terminated, truncated to name_len), launch count and summed
 * milliseconds of the index-th kernel name (alphabetical); ACSC_EINVAL past
 * the last one.  Timing serialises nothing but adds two event records per
 * launch.  acsc_stats_only(tag) restricts timing to the launches of that
 * kernel name (copied; NULL or "" times every launch again), so that one
 * kernel can be timed inside a loop without the records of all the others;
 * it keeps the counters.  Returns ACSC_EINVAL for a name of 64 or more
 * characters. */
int acsc_stats_enable(int on);
int acsc_stats_only(const char *tag);
int acsc_stats_read(int index, char *name, size_t name_len, int64_t *launches, double *total_ms);

/* ------------------------------------------------------------------------
 * Activation-masking compressor (paper Sec. 3.1; Alg. 1; App. F).
 *
 * The mask of a [B, S, H] hidden state at one pipeline boundary is the
 * paper's shared pseudorandom function g(layer, step, B, S, H): sender and
 * receiver rebuild it from this key, so only the kept values need to cross
 * the link.  The backward pass uses the same key, so the activation gradient
 * is packed at exactly the positions kept in the forward pass.  The key has
 * no direction field on purpose.
 *
 * Per token row r = b*S + s the kept set I_r holds K distinct indices of
 * [0, H) in ascending order; it is the image of [0, K) under a keyed Feistel
 * permutation of [0, H) (cycle walking), keyed by mix64 over the fields
 * below.  The full construction is specified in the project's design notes
 * and implemented independently by the CPU oracle.
 * ---------------------------------------------------------------------- */
typedef struct ac_mask_key {
    uint64_t seed;        /* run-wide secret shared by sender and receiver   */
    uint64_t step;        /* optimisation step t                             */
    uint32_t layer;       /* boundary layer index l                          */
    uint32_t microbatch;  /* microbatch id within the step                   */
    uint32_t B, S, H;     /* tensor shape: batch, sequence length, hidden    */
} ac_mask_key;

/* K = round(keep * H) kept dimensions per token (Sec. 3.1, keep = 1 - p),
 * computed as floor(keep*H + 0.5) in double.  Requires 1 <= H <= 65536,
 * 0 < keep <= 1 and a result in [1, H]; else ACSC_EINVAL. */
int ac_keep_count(int H, double keep, int *K);

/* Pack (Sec. 3.1 forward send; Alg. 1 backward send, same key):
 *   vals[r, i] = x[r, I_r[i]]   (bit copy)     for 0 <= r < rows, 0 <= i < K
 *   idx[r, i]  = I_r[i]         (if idx != NULL)
 * x     device, [rows, ld_x] elements of `dt`, ld_x >= H.
 * vals  device, [rows, K] contiguous, same dtype; must not overlap x.
 * idx   device or NULL, [rows, K] uint16, ascending within each row.
 * Requires rows == key->B * key->S, H == key->H, 1 <= K <= H <= 65536, and
 * element-size alignment of x and vals (2-byte idx). */
int ac_mask_pack(const void *x, acsc_dtype dt, int64_t rows, int H, int64_t ld_x, int K,
                 const ac_mask_key *key, void *vals, uint16_t *idx, hipStream_t stream);

/* Unpack and scatter (Sec. 3.1 receiver; App. F receiver-side rescale):
 *   y[r, j] = round(scale * vals[r, i])  if j = I_r[i]
 *   y[r, j] = +0                          otherwise,     for j < H
 * The product is rounded once to `dt` (nearest even), so scale = 1 copies
 * bits exactly (for bf16, products in the fp32 normal range).  scale = H/K
 * makes the fixed-K mask unbiased; the paper's 1/(1-p) is within 0.5% of it.
 * vals  device, [rows, K] contiguous.
 * idx   device or NULL.  NULL: positions are rebuilt from `key` (the paper's
 *       wire format).  Otherwise row r of idx must be strictly ascending, as
 *       ac_mask_pack writes it; entries >= H are ignored.
 * y     device, [rows, ld_y], ld_y >= H; columns >= H are not touched; must
 *       not overlap vals or idx.
 * Same shape and key requirements as ac_mask_pack. */
int ac_unpack_scatter(const void *vals, const uint16_t *idx, acsc_dtype dt, int64_t rows, int H,
                      int K, const ac_mask_key *key, float scale, void *y, int64_t ld_y,
                      hipStream_t stream);

/* Batched forms over nlayers pipeline boundaries in one launch (Alg. 1: the
 * boundary after layer l has its own mask M_l = g(l, t, B, S, H); Sec. 3.1).
 * Boundary l (0 <= l < nlayers) is keyed exactly as the single call with
 * key->layer + l, and its tensors start at base + l * stride, strides counted
 * in elements of the array they step:
 *   x / y      [rows, ld] of dt per boundary, stride x_stride / y_stride;
 *   vals       [rows, K] contiguous per boundary, stride vals_stride;
 *   idx_in, idx_out   [rows, K] uint16 per boundary, stride idx_stride.
 * Each boundary's result is bit-identical to the single call on its tensors.
 *
 * Index lists let each stage evaluate a boundary's mask once (the paper's
 * shared PRF: both stages rebuild it, neither sends it):
 *   pack   idx_in == NULL: the mask comes from the key; idx_out (or NULL)
 *          receives the kept positions (what ac_mask_pack writes to idx).
 *          idx_in != NULL: vals[r, i] = x[r, idx_in[r, i]] (bit copies; an
 *          entry >= H gives +0) and the key's fields other than layer are
 *          only checked; idx_out must then be NULL.
 *   unpack idx_in == NULL: positions from the key; idx_out (or NULL)
 *          receives them.  idx_in != NULL: as ac_unpack_scatter with idx
 *          (strictly ascending rows; entries >= H ignored); idx_out NULL.
 * So the sender packs from the key writing idx_out and later unpacks the
 * gradient from those lists, and the receiver unpacks from the key writing
 * idx_out and packs the gradient from them: only the values cross the link.
 * Requirements as the single calls, plus 0 <= nlayers <= 65535 (0 is a
 * no-op), key->layer + nlayers - 1 < 2^32, non-negative input strides, and
 * output strides that keep boundaries apart when nlayers > 1:
 * vals_stride >= rows * K, idx_stride >= rows * K (with idx_out),
 * y_stride >= (rows - 1) * ld_y + H.  16-byte stores are used only when
 * every boundary's rows are 16-byte aligned. */
int ac_mask_pack_batched(const void *x, acsc_dtype dt, int nlayers, int64_t rows, int H, int64_t ld_x,
                         int64_t x_stride, int K, const ac_mask_key *key, void *vals, int64_t vals_stride,
                         const uint16_t *idx_in, uint16_t *idx_out, int64_t idx_stride,
                         hipStream_t stream);
int ac_unpack_scatter_batched(const void *vals, int64_t vals_stride, acsc_dtype dt, int nlayers, int64_t rows,
                              int H, int K, const ac_mask_key *key, const uint16_t *idx_in, uint16_t *idx_out,
                              int64_t idx_stride, float scale, void *y, int64_t ld_y, int64_t y_stride,
                              hipStream_t stream);

/* ------------------------------------------------------------------------
 * Bernoulli mask variant (App. F: every entry of the mask an independent
 * Bernoulli draw, kept with probability 1 - p; the receiver rescales by
 * 1 / (1 - p)).  Rows keep a variable number of entries, so the payload is
 * laid out by row offsets: row r owns vals[row_ptr[r] .. row_ptr[r + 1]),
 * its kept entries in ascending position order.
 * The per-entry draw (our specification; the paper gives no PRF): with k_r
 * the row key of the fixed-K mask (the same key chain), a and b its low and
 * high 32 bits, entries 2q and 2q + 1 of the row take the low and the high 16
 * bits of fmix32(fmix32(a ^ q) ^ b), and are kept when those are below
 * T = floor(keep * 65536 + 0.5) (inclusion probability T / 65536).
 * ---------------------------------------------------------------------- */

/* The mask of a [rows, H] tensor for `key`, computed once and reused by
 * every pack and unpack with that key (both directions of a boundary):
 *   row_ptr  device int64 [rows + 1] out: row_ptr[0] = 0, row_ptr[r + 1] -
 *            row_ptr[r] = entries kept in row r; row_ptr[rows] = nnz.
 *   bits     device uint32 [rows, ceil(H / 32)] out: bit j % 32 of word
 *            j / 32 of row r is set iff entry (r, j) is kept.
 * Requires 0 < keep <= 1 with T >= 1, 1 <= H <= 65536, key->H == H,
 * key->B * key->S == rows, 8-byte aligned row_ptr, 4-byte aligned bits.
 * The sender and the receiver compute the same row_ptr and bits from the
 * key alone; nothing but the values needs to cross the link. */
int ac_bern_mask(int64_t rows, int H, double keep, const ac_mask_key *key, int64_t *row_ptr,
                 uint32_t *bits, hipStream_t stream);

/* Pack: vals[row_ptr[r] + i] = x[r, j_i] (bit copies) for the kept entries
 * j_0 < j_1 < ... of row r; idx (device uint16 or NULL) gets the j_i.
 * x     device [rows, ld_x] of dt (ld_x >= H).
 * vals  device, capacity `cap` elements (size it by row_ptr[rows]); slots
 *       at or past cap are not written.
 * row_ptr, bits  from ac_bern_mask for the same rows, H and key. */
int ac_bern_pack(const void *x, acsc_dtype dt, int64_t rows, int H, int64_t ld_x,
                 const int64_t *row_ptr, const uint32_t *bits, void *vals, uint16_t *idx,
                 int64_t cap, hipStream_t stream);

/* Unpack: y[r, j] = round(scale * vals[row_ptr[r] + i]) at the i-th kept
 * entry j of row r, +0 elsewhere (columns >= H untouched).  The product is
 * rounded once (as ac_unpack_scatter).  Slots at or past cap read as zero.
 * y device [rows, ld_y], ld_y >= H, must not overlap vals. */
int ac_bern_unpack(const void *vals, acsc_dtype dt, int64_t rows, int H, const int64_t *row_ptr,
                   const uint32_t *bits, int64_t cap, float scale, void *y, int64_t ld_y,
                   hipStream_t stream);

/* ------------------------------------------------------------------------
 * Spectral corrector (paper Sec. 3.2; Alg. 1; App. E).
 * ---------------------------------------------------------------------- */

/* Largest supported k = r + oversample (columns of the subspace iteration). */
#define SC_KMAX 192

/* Bytes of device workspace that sc_build_prior and sc_correct need for an
 * m x n matrix, prior rank r and oversampling p (k = min(r + p, m, n)).
 * Requires 1 <= r <= min(m, n, SC_KMAX), p >= 0. */
int sc_workspace_size(int m, int n, int r, int oversample, acsc_dtype dt, size_t *bytes);

/* Anchor prior (Sec. 3.2; Alg. 1 on anchor arrival; App. E):
 *   1. if G_anc != NULL:  M <- beta * M + (1 - beta) * G_anc       (EMA)
 *   2. (U, s, V) = the top-r singular triplets of M                 (SVD)
 *   3. d_i = s_i / (s_i + tau), with 0/0 taken as 0                 (filter)
 * The SVD is computed by randomised block subspace iteration on the device:
 * k = min(r + oversample, m, n) columns, `power_iters` passes of M^T then M,
 * CholeskyQR2 re-orthonormalisation, Rayleigh-Ritz via one-sided Jacobi.
 * Starting block: V_warm (n x r, e.g. the previous V) padded with random
 * columns drawn from `seed`, or all random when V_warm is NULL.
 * G_anc  device or NULL, [m, n] of `dt`.
 * M      device fp32 [m, n], in/out (the EMA state; start it at zero).
 * U      device fp32 [m, r] out, orthonormal columns.
 * s, d   device fp32 [r] out; s descending, d in [0, 1).
 * V      device fp32 [n, r] out, orthonormal columns.
 * Singular values at or below 1e-5 times the largest (the numerical rank of
 * an fp32 iteration; M of rank < r) are returned as s_i = d_i = 0 with zero
 * columns in U and V.
 * Requires 0 <= beta <= 1, tau >= 0, power_iters >= 0, 1 <= r <= min(m,n,SC_KMAX),
 * ws_bytes >= sc_workspace_size(...), 256-byte aligned ws. */
int sc_build_prior(const void *G_anc, acsc_dtype dt, float *M, int m, int n, float beta, int r,
                   int oversample, int power_iters, float tau, const float *V_warm, uint64_t seed,
                   float *U, float *s, float *V, float *d, void *ws, size_t ws_bytes,
                   hipStream_t stream);

/* Spectral correction of one masked weight gradient (Sec. 3.2; Alg. 1):
 *   X = U^T G V;  X_f = diag(d) X diag(d);  G_filt = U X_f V^T;
 *   G_proj = alpha * G + (1 - alpha) * G_filt
 * G       device [m, n] of `dt`.
 * U, V    device fp32 [m, r], [n, r];  d device fp32 [r].
 * G_proj  device [m, n] of `dt`; may equal G (in place), must not partially
 *         overlap it.
 * Accumulation is fp32.  For bf16 G the products run on bf16 matrix cores,
 * with U X_f and V rounded to bf16 (relative error ~1e-3, well inside the
 * 2e-2 budget of bf16 inputs); for fp32 G everything stays fp32.
 * Requires 1 <= r <= SC_KMAX, r <= min(m, n), ws as for sc_build_prior,
 * element-aligned pointers. */
int sc_correct(const void *G, acsc_dtype dt, int m, int n, const float *U, const float *d,
               const float *V, int r, float alpha, void *G_proj, void *ws, size_t ws_bytes,
               hipStream_t stream);

/* sc_correct without a workspace argument, for callers that cannot allocate
 * device memory (code under HIP graph capture, serving loops that forbid
 * allocation).  Its scratch is a device array of SC_STATIC_SCRATCH_BYTES
 * inside the library: each device that runs this call holds its own copy
 * until the process ends, and its address is looked up once per device on
 * the first call there.  The call allocates no device memory.  Every call on
 * one device shares that device's array and leaves its contents behind (the
 * correction writes every scratch byte it reads first, so nothing carries
 * from one call to the next): calls that may overlap on one device, on
 * different streams or threads, race and must be ordered by the caller.
 * Arguments, results and errors as sc_correct; a shape whose scratch
 * (sc_adamw_workspace_size) exceeds SC_STATIC_SCRATCH_BYTES returns
 * ACSC_ENOSPC before anything is enqueued.  96 MiB covers a 28672 x 8192
 * bf16 matrix at r = 128 (88 MiB). */
#define SC_STATIC_SCRATCH_BYTES (96u * 1024u * 1024u)
int sc_correct_static(const void *G, acsc_dtype dt, int m, int n, const float *U, const float *d,
                      const float *V, int r, float alpha, void *G_proj, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Batched forms: the same operations on several weight matrices (e.g. all
 * targeted matrices of the layers a pipeline stage holds) in one call.  Every
 * kernel is launched once for up to 16 matrices, so the latency-bound small
 * steps (Cholesky, Jacobi) of different matrices run side by side, and the
 * streaming passes of small matrices fill the GPU together.
 * ---------------------------------------------------------------------- */
typedef struct sc_matrix {
    const void *G;          /* build: G_anc [m, n] of dt, or NULL (no arrival);
                               correct: the masked gradient G [m, n] of dt     */
    float *M;               /* build: EMA state, fp32 [m, n], in/out; unused by correct */
    int m, n;               /* shape of this matrix                              */
    float *U, *s, *V, *d;   /* build: outputs; correct: the prior (s unused)     */
    const float *V_warm;    /* build: optional [n, r] start block, or NULL       */
    void *G_proj;           /* correct: output [m, n] of dt (may equal G); unused by build */
    void *ws;               /* device workspace of this matrix (256-byte aligned) */
    size_t ws_bytes;        /* >= sc_workspace_size(m, n, r, oversample, dt)     */
} sc_matrix;

/* sc_build_prior on each of mats[0 .. count-1] with shared dt, beta, r,
 * oversample, power_iters and tau; matrix i starts from the random block of
 * seed + i.  Matrices must not share M, outputs or workspaces.  All arguments
 * of all matrices are checked before anything is enqueued. */
int sc_build_prior_batched(int count, const sc_matrix *mats, acsc_dtype dt, float beta, int r,
                           int oversample, int power_iters, float tau, uint64_t seed,
                           hipStream_t stream);

/* The same batched build in its two phases, for a caller that wants other
 * work beside the second (App. E's top-r SVD as a randomised subspace
 * iteration followed by a Rayleigh-Ritz step):
 *   sc_build_subspace_batched: the EMA of Sec. 3.2, the power passes and
 *     the last product Z = M^T Q, all streaming M; it leaves Q and Z in each
 *     matrix's workspace and writes no output;
 *   sc_build_ritz_batched: the Rayleigh-Ritz step on Z (a k x k Gram, its
 *     Cholesky factor and that factor's SVD on a few workgroups, then the
 *     basis U, V, s and the filter d); it does not touch M.
 * Both take exactly the arguments of sc_build_prior_batched, and the ritz
 * call must follow the subspace call with the same arguments and
 * workspaces, in stream order, with nothing writing those workspaces in
 * between.  The ritz call reads neither G_anc nor beta, power_iters or seed.
 * The pair enqueues the same kernels in the same order as one
 * sc_build_prior_batched call, so the results are bit-identical.  Errors as
 * for sc_build_prior_batched. */
int sc_build_subspace_batched(int count, const sc_matrix *mats, acsc_dtype dt, float beta, int r,
                              int oversample, int power_iters, float tau, uint64_t seed,
                              hipStream_t stream);
int sc_build_ritz_batched(int count, const sc_matrix *mats, acsc_dtype dt, float beta, int r,
                          int oversample, int power_iters, float tau, uint64_t seed,
                          hipStream_t stream);

/* Status of the last build on each matrix's workspace (App. E's top-r SVD:
 * the Rayleigh-Ritz step ends with a one-sided Jacobi SVD run to a
 * tolerance, at most 40 sweeps).  Synchronises `stream`, then reads the
 * status words the build left at the head of each workspace (mats[i].ws;
 * the other fields are not read).  Returns ACSC_OK when every matrix's
 * Jacobi met its tolerance; ACSC_ENOCONV when one stopped at the sweep cap
 * above it, or when a Rayleigh-Ritz phase ran without a subspace phase
 * having stamped that workspace since the last Rayleigh-Ritz phase (e.g.
 * sc_build_ritz_batched alone, or after a correction that reused the
 * workspace); acsc_last_error() names the first such matrix.  sweeps and
 * residual (arrays of count, or NULL) receive each matrix's sweeps used and
 * its last sweep's largest off-diagonal ratio.  ACSC_ENOCONV also reports
 * a subspace phase whose fused EMA pass (bf16 shadow, large batches) gave up
 * one of its bounded waits between the waves of a workgroup (the wait polls
 * for about a second or more before it gives up; the kernel then finishes
 * with a product that is not to be trusted).  A workspace that never held
 * a build gives unspecified values.  The environment variables
 * ACSC_JACOBI_MAX_SWEEPS and ACSC_EMA_SPIN_LIMIT, read by each build call,
 * lower the sweep cap (1..40) and the polls of a wait (0 gives up at the
 * first unmet check), so that both reports can be produced on purpose. */
int sc_build_status(int count, const sc_matrix *mats, int *sweeps, float *residual, hipStream_t stream);

/* sc_correct on each of mats[0 .. count-1] with shared dt, r and alpha. */
int sc_correct_batched(int count, const sc_matrix *mats, acsc_dtype dt, int r, float alpha,
                       hipStream_t stream);

/* ------------------------------------------------------------------------
 * Corrected AdamW step (Alg. 1: the fast weights are updated by AdamW on
 * G_proj; App. I: AdamW, betas (0.9, 0.999), gradient norm clipped at 0.2).
 * The correction and the update run as one step: G_proj is never written to
 * device memory.
 * ---------------------------------------------------------------------- */

/* Optimiser state of one weight matrix: device fp32 arrays of the matrix's
 * [m, n] shape (row-major), read and written in place; the first and second
 * moments start at zero.  16-byte aligned arrays (with n % 8 == 0) take the
 * vectorised path; 4-byte alignment is required. */
typedef struct sc_adamw_state {
    float *W;     /* weights                    */
    float *m1;    /* first moment (Adam's m_t)  */
    float *m2;    /* second moment (Adam's v_t) */
} sc_adamw_state;

/* Hyperparameters of one step (shared by every matrix of a call). */
typedef struct sc_adamw_hparams {
    float lr;             /* this step's learning rate (any schedule is the caller's) */
    float beta1, beta2;   /* moment decay rates, each in [0, 1)                        */
    float eps;            /* > 0, added to the bias-corrected sqrt(m2)                 */
    float weight_decay;   /* >= 0, decoupled: W <- W (1 - lr * weight_decay)           */
    int64_t step;         /* t >= 1: bias corrections 1 - beta^t                       */
    float max_norm;       /* > 0: global-norm clipping at max_norm; <= 0: none          */
} sc_adamw_hparams;

/* Bytes of workspace sc_correct_adamw_batched needs per matrix (it is also
 * covered by sc_workspace_size for the same shape, so one workspace serves the
 * build, the correction and this step). */
int sc_adamw_workspace_size(int m, int n, int r, acsc_dtype dt, size_t *bytes);

/* For every matrix i of the call (mats[i] as for sc_correct_batched, except
 * that G_proj is unused and may be NULL; states[i] its optimiser state):
 *   G_proj_i = alpha G_i + (1 - alpha) U_i diag(d) (U_i^T G_i V_i) diag(d) V_i^T
 *   N        = sqrt(sum_i ||G_proj_i||_F^2)            (the call's global norm)
 *   c        = min(1, max_norm / (N + 1e-6))  if max_norm > 0, else 1
 *   g        = c G_proj_i
 *   W  <- W (1 - lr wd);  m1 <- beta1 m1 + (1 - beta1) g;  m2 <- beta2 m2 + (1 - beta2) g^2
 *   W  <- W - lr (m1 / (1 - beta1^t)) / (sqrt(m2 / (1 - beta2^t)) + eps)
 * The decoupled weight decay is that of AdamW (Loshchilov & Hutter 2019);
 * the clipping that of the common global-norm form.  N is formed as
 * alpha^2 ||G||^2 + 2 alpha (1 - alpha) <X, X_f> + (1 - alpha)^2 ||X_f||^2,
 * which holds for the orthonormal U, V of sc_build_prior.
 * norm_out  device fp32 scalar or NULL: receives N (before clipping).
 * The state arrays of different matrices must not overlap; G is only read.
 * Arithmetic is fp32 (as sc_correct for the blend).  All arguments of all
 * matrices are checked before anything is enqueued; errors as elsewhere. */
int sc_correct_adamw_batched(int count, const sc_matrix *mats, const sc_adamw_state *states,
                             acsc_dtype dt, int r, float alpha, const sc_adamw_hparams *hp,
                             float *norm_out, hipStream_t stream);

/* ------------------------------------------------------------------------
 * PowerSGD compressor with error feedback, one worker's share (the
 * data-parallel side the method is paired with: Sec. 3.3, Sec. 5 setup,
 * App. J family F3; Vogels, Karimireddy & Jaggi 2019, rank-r compression
 * and error-feedback SGD).  One step on a matrix:
 *   psgd_project:      M = G + E (stored in E);  P = M Q
 *   (across workers:   P <- mean of P over the workers)
 *   psgd_orthogonalize: P <- orth(P) (Gram-Schmidt order, here CholeskyQR2);
 *                      Q <- M^T P
 *   (across workers:   Q <- mean of Q over the workers)
 *   psgd_decompress:   out = P Q^T (in dt);  E <- M - out
 * On one worker the means are the identity and psgd_step runs the three
 * phases.  Q carries over to the next step (warm start); the caller draws
 * the first Q (e.g. Gaussian) and zeroes E once.  The factors of a matrix
 * are m r + n r numbers against m n: rank r = floor(m n / (64 (m + n)))
 * compresses by at least x64.
 * ---------------------------------------------------------------------- */
typedef struct psgd_matrix {
    const void *G;    /* [m, n] gradient of dt, row-major; 16-byte aligned       */
    float *E;         /* [m, n] fp32 memory, in/out; 16-byte aligned; holds M
                         from psgd_project until psgd_decompress                 */
    float *P;         /* [m, r] fp32: P = M Q (project), then P_hat (orthogonalize) */
    float *Q;         /* [n, r] fp32: previous Q (project), then M^T P_hat          */
    void *out;        /* [m, n] of dt: the decompressed gradient; may equal G,
                         must not overlap E, P, Q or the workspace                */
    int m, n;
    void *ws;         /* device workspace (256-byte aligned); carries the bf16
                         copy of M from psgd_project to psgd_orthogonalize: keep
                         it for this matrix in between                            */
    size_t ws_bytes;  /* >= psgd_workspace_size(m, n, r, dt)                      */
} psgd_matrix;

/* Bytes of workspace a psgd call needs for one m x n matrix at rank r.
 * Requires 1 <= r <= min(m, n, SC_KMAX). */
int psgd_workspace_size(int m, int n, int r, acsc_dtype dt, size_t *bytes);

/* The phases and the whole step over mats[0 .. count-1] (shared dt and r).
 * Arithmetic: fp32 memory and accumulation; for bf16 G the two projections
 * run on bf16 matrix cores from a bf16 copy of M and of the thin factor, the
 * Gram matrices of CholeskyQR2 in fp64, and out = bf16(P Q^T) from bf16 P
 * and Q; for fp32 G everything stays fp32.  E is taken against out as
 * stored, so what out loses to rounding is carried to the next step.  A
 * column of P that is numerically dependent on the earlier ones (Cholesky
 * pivot at or below 1e-15 r times the largest diagonal of P^T P) becomes
 * zero, as does the matching column of Q.  Matrices must not share any
 * buffer or workspace; all arguments are checked before anything is
 * enqueued; errors as elsewhere. */
int psgd_project(int count, const psgd_matrix *mats, acsc_dtype dt, int r, hipStream_t stream);
int psgd_orthogonalize(int count, const psgd_matrix *mats, acsc_dtype dt, int r, hipStream_t stream);
int psgd_decompress(int count, const psgd_matrix *mats, acsc_dtype dt, int r, hipStream_t stream);
int psgd_step(int count, const psgd_matrix *mats, acsc_dtype dt, int r, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* ACSC_H */
