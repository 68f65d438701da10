/*
 * eogp.h -- C ABI of the EOGP hot path (eigenbasis-corrected one-bit gradient
 * projection) on AMD Instinct MI355X (gfx950).
 *
 * The path has two parts. Storing: each example's per-module gradient
 * G = sum_t ds_t a_t^T is rotated into the K-FAC Kronecker eigenbasis
 * Q_A (x) Q_S one token at a time, the coordinates with the m largest
 * corrected eigenvalues are kept and half-whitened (first stage), projected by
 * the PCA matrix P (second stage) and stored as packed sign bits plus one fp16
 * scale. Scoring: unquantized query coordinates are scored against the stored
 * codes and a per-query top-k is kept.
 *
 * Conventions for every call:
 *   - Array arguments are DEVICE pointers owned by the caller unless a comment
 *     says "host". The library never frees caller memory. Only
 *     eogp_plan_create allocates (the plan's own memory, released by
 *     eogp_plan_destroy); scratch for the other calls comes from a caller
 *     workspace whose size the matching *_workspace_size call returns.
 *   - Arrays are row-major and contiguous unless a leading dimension ("ld",
 *     in elements) or a row stride is given.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream). Calls
 *     only enqueue work on it and return, except eogp_plan_create, the
 *     one-shot eogp_rotate_retain and eogp_pca_fit, which synchronise `stream`
 *     once. Host arrays passed to an enqueuing call (such as k_per_module)
 *     are read before the call returns and may be released at once. The
 *     enqueuing calls launch kernels only (eogp_plan_copy_retained a
 *     device-to-device copy): no allocation, memset or host wait, so a
 *     sequence of them can be captured in a HIP graph and replayed.
 *   - Argument errors return EOGP_ERR_INVALID before anything is enqueued;
 *     EOGP_ERR_UNSUPPORTED marks a valid but unimplemented dtype/shape mix;
 *     EOGP_ERR_DEVICE a HIP launch or runtime error; EOGP_ERR_WORKSPACE a
 *     workspace smaller than required. eogp_last_error() describes the last
 *     failure on the calling thread.
 */
#ifndef EOGP_H
#define EOGP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t eogp_status;
#define EOGP_OK 0
#define EOGP_ERR_INVALID (-1)
#define EOGP_ERR_UNSUPPORTED (-2)
#define EOGP_ERR_DEVICE (-3)
#define EOGP_ERR_WORKSPACE (-4)

typedef enum { EOGP_F32 = 0, EOGP_BF16 = 1, EOGP_F16 = 2 } eogp_dtype;

/* Arithmetic of the dense contractions. FAST: one MFMA pass on operands
 * rounded to bf16 (or fp16 where an operand is given in fp16), fp32
 * accumulation. ACCURATE: every fp32 operand is split into a high and a low
 * 16-bit part and the cross products are accumulated in fp32 (three MFMA
 * passes when both operands are fp32, two when one is already 16-bit), which
 * carries about 16 significant bits into each product. F16 (first stage and
 * EK-FAC pass): one MFMA pass on operands rounded once to fp16 (11
 * significant bits, 8 times finer than bf16), fp32 accumulation; inputs are
 * first multiplied by the plan's power-of-two exponents (see
 * eogp_plan_set_input_exponents) so they sit inside fp16's normal range
 * (2^-14 <= |x| < 65504). bf16 inputs enter this mode exactly inside that
 * range (8 significant bits fit in fp16's 11); only the bases and the rotated
 * tokens are rounded. */
typedef enum { EOGP_PREC_FAST = 0, EOGP_PREC_ACCURATE = 1, EOGP_PREC_F16 = 2 } eogp_prec;

/* ------------------------------------------------------------------------
 * Fitting shared projections: retained-axis selection (Algorithm 1, fitting
 * block: the axes with the m_u largest corrected eigenvalues are kept;
 * Section 3.2 first stage and eq. sigma_ekfac, which makes the m largest
 * corrected eigenvalues the top-m PCA axes of Sigma_proxy).
 *
 * A plan holds, for one module, the m retained axes in canonical order
 * (Lambda descending, then flat index j*d_in + k ascending), their
 * half-whitening weights (Lambda_r + lambda)^-1/2 (eq. first_stage), and the
 * eigenvector columns of Q_A and Q_S those axes use, gathered so the first
 * stage runs as dense contractions without forming Q_m (eq.
 * app_projection_maps: the map is stored as its two Kronecker factors plus
 * the indices of the kept coordinates).
 *
 *   eigvals  [d_out, d_in] fp32: corrected eigenvalue Lambda[j, k] of the
 *            axis Q_A[:, k] (x) Q_S[:, j] (eq. ekfac_eigendecompose).
 *   damping  lambda > 0.
 *   m        1 <= m <= d_in * d_out.
 *   Q_A      [d_in, d_in] fp32, column k = k-th eigenvector of A = E[a a^T].
 *   Q_S      [d_out, d_out] fp32, column j = j-th eigenvector of S.
 *   out      receives the plan (host handle).
 * Errors: EOGP_ERR_INVALID for bad sizes, NULL pointers, damping <= 0, a NaN
 * anywhere in eigvals, or a retained Lambda_r + lambda <= 0. Runs on `stream`
 * and synchronises it once (it reads back the retained-set sizes).
 * ------------------------------------------------------------------------ */
typedef struct eogp_plan eogp_plan;

typedef struct {
  int64_t d_out, d_in, m;
  double damping;
  int64_t n_rows;   /* |J|: distinct Q_S columns used by the retained set   */
  int64_t n_cols;   /* |K|: distinct Q_A columns used by the retained set   */
  int64_t n_tiles;  /* 32 x 32 blocks of (row, column) pairs holding retained axes */
  const int32_t* retained_flat;    /* device [m]: j*d_in + k, canonical order */
  const float* retained_weight;    /* device [m]: (Lambda_r + lambda)^-1/2     */
} eogp_plan_info;

eogp_status eogp_plan_create(const float* eigvals, int64_t d_out, int64_t d_in,
                             double damping, int64_t m, const float* Q_A,
                             const float* Q_S, void* stream, eogp_plan** out);
void eogp_plan_destroy(eogp_plan* plan);
eogp_status eogp_plan_get_info(const eogp_plan* plan, eogp_plan_info* info);
/* Copy the retained axes (flat index j*d_in + k, int32 [m]) and their
 * half-whitening weights (fp32 [m]) into caller device buffers; either output
 * may be NULL. Enqueued on `stream`. */
eogp_status eogp_plan_copy_retained(const eogp_plan* plan, int32_t* flat_out,
                                    float* weight_out, void* stream);
/* Power-of-two input scaling of the plan's EOGP_PREC_F16 first stage:
 * activations are multiplied by 2^e_acts and output-gradients by 2^e_grads
 * before they are rounded to fp16, and every coordinate by
 * 2^-(e_acts + e_grads) afterwards. The first stage is bilinear in (a, ds),
 * so the result is unchanged up to fp16 rounding; the exponents only move
 * the inputs into fp16's range (e.g. e_grads = 10 for gradients of order
 * 1e-5). Both default to 0. Errors: EOGP_ERR_INVALID for a NULL plan or an
 * exponent outside [-60, 60]. Host-only; affects later calls. */
eogp_status eogp_plan_set_input_exponents(eogp_plan* plan, int32_t e_acts, int32_t e_grads);

/* ------------------------------------------------------------------------
 * First stage (eq. first_stage; eq. app_projection_maps; Algorithm 1,
 * storing: x_{i,u} <- T_u(L_u g_{i,u})). For every example i:
 *   Z[i, r] = (Lambda_r + lambda)^-1/2
 *             * sum_{t : token_mask[i, t] != 0} (Q_S[:, j_r] . ds[i, t])
 *                                               (Q_A[:, k_r] . a[i, t])
 * for the retained axes r = 0..m-1 of the plan, in canonical order. The
 * gradient is never formed: valid tokens are compacted, rotated onto the
 * needed eigenvectors with MFMA contractions, and the retained products are
 * summed per example (the loss is token-summed over valid positions).
 *
 *   acts       [N, T, d_in]  in `in_dtype` (EOGP_F32 or EOGP_BF16); token
 *              (i, t) starts at element (i*T + t) * ld_acts (ld_acts >= d_in,
 *              or 0 for d_in). Rows whose byte offset is a multiple of 16 take
 *              the fast load path (fp32: ld_acts % 4 == 0; bf16: % 8 == 0);
 *              16-bit rows must satisfy it.
 *   out_grads  [N, T, d_out] in `in_dtype`, token stride ld_grads likewise.
 *   token_mask [N, T] uint8, or NULL for all tokens valid. Masked tokens are
 *              never read and may hold anything, NaN included.
 *   Z          [N, ldz] fp32, ldz >= m; columns m..ldz-1 are not written.
 *   prec       EOGP_PREC_ACCURATE keeps about 16 bits per product;
 *              EOGP_PREC_F16 rounds inputs and bases once to fp16 (relative
 *              error of a row of Z about 5e-4 for inputs inside fp16's normal
 *              range, fp32 or bf16); EOGP_PREC_FAST rounds operands to bf16
 *              and keeps the rotated tokens in bf16 (about 3e-3).
 *   ws         workspace of at least eogp_rotate_retain_workspace_size bytes.
 * Sizes: N*T + 8N + 256 < 2^31 (the compacted token list is indexed in
 * 32 bits), else EOGP_ERR_INVALID.
 * ------------------------------------------------------------------------ */
size_t eogp_rotate_retain_workspace_size(const eogp_plan* plan, int64_t N, int64_t T);
/* The planned call takes the plan built once per module (eogp_plan_create)
 * and writes Z in `z_dtype`: EOGP_F32, or EOGP_F16, each coordinate rounded
 * once to fp16 (nearest even; beyond fp16's range it becomes inf) -- the
 * paper caches first-stage coordinates in FP16, and eogp_pca_project takes
 * such a Z directly. Other z_dtype values give EOGP_ERR_INVALID. */
eogp_status eogp_rotate_retain_planned(const eogp_plan* plan, const void* acts,
                                       int64_t ld_acts, const void* out_grads,
                                       int64_t ld_grads, eogp_dtype in_dtype,
                                       const uint8_t* token_mask, int64_t N, int64_t T,
                                       void* Z, eogp_dtype z_dtype, int64_t ldz,
                                       eogp_prec prec, void* ws, size_t ws_bytes,
                                       void* stream);

/* The valid-token list shared by every module of a batch (Algorithm 1 runs
 * per example; all linear modules of an example see the same token mask).
 * eogp_compact_tokens writes the list for (token_mask, N, T) into the head of
 * a first-stage workspace: eogp_compact_tokens_workspace_size(N, T) bytes
 * (0 for invalid sizes), which every eogp_rotate_retain_workspace_size for
 * the same N and T includes. `prec` selects the list's layout: runs of each
 * example padded to 8 tokens for EOGP_PREC_F16 and EOGP_PREC_FAST, packed for
 * EOGP_PREC_ACCURATE. eogp_rotate_retain_compacted then runs the planned first
 * stage of one module without compacting again; its arguments are those of
 * eogp_rotate_retain_planned without the mask, and ws must hold the list
 * written for the same N, T and a `prec` of the same layout (the list is not
 * checked: another list gives wrong coordinates, with every access inside
 * the workspace and the token rows). Sizes and errors as for the planned
 * call; both calls only enqueue work. */
size_t eogp_compact_tokens_workspace_size(int64_t N, int64_t T);
eogp_status eogp_compact_tokens(const uint8_t* token_mask, int64_t N, int64_t T, eogp_prec prec,
                                void* ws, size_t ws_bytes, void* stream);
eogp_status eogp_rotate_retain_compacted(const eogp_plan* plan, const void* acts,
                                         int64_t ld_acts, const void* out_grads,
                                         int64_t ld_grads, eogp_dtype in_dtype, int64_t N,
                                         int64_t T, void* Z, eogp_dtype z_dtype, int64_t ldz,
                                         eogp_prec prec, void* ws, size_t ws_bytes,
                                         void* stream);

/* One-shot form with the paper's arguments: builds a plan from
 * (eigvals, damping, m, Q_A, Q_S), runs the first stage, releases the plan.
 * Synchronises `stream`. Workspace: eogp_rotate_retain_oneshot_workspace_size
 * (an upper bound for any plan of these shapes; 0 for invalid sizes). */
size_t eogp_rotate_retain_oneshot_workspace_size(int64_t N, int64_t T, int64_t d_in,
                                                 int64_t d_out, int64_t m);
eogp_status eogp_rotate_retain(const void* acts, int64_t ld_acts, const void* out_grads,
                               int64_t ld_grads, eogp_dtype in_dtype,
                               const uint8_t* token_mask,
                               int64_t N, int64_t T, int64_t d_in, int64_t d_out,
                               const float* Q_A, const float* Q_S, const float* eigvals,
                               double damping, int64_t m, float* Z, int64_t ldz,
                               eogp_prec prec, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Second stage (eq. second_stage; Appendix E.3, implementation and runtime:
 * one correction matrix applied to a whole batch of cached first-stage
 * coordinates):
 *   X[i, c] = sum_r Z[i, r] P[r, c],  i.e. x_i = P^T z_i.
 *
 *   Z   [N, ldz] in `z_dtype` (first m columns used): EOGP_F32 with any P, or
 *       16-bit Z of P's own type (EOGP_F16 with fp16 P, EOGP_BF16 with bf16 P;
 *       rows on 16-byte boundaries: ldz % 8 == 0, Z 16-byte aligned), else
 *       EOGP_ERR_UNSUPPORTED. A 16-bit Z enters one MFMA product as it is.
 *   P   the m x k PCA matrix stored COLUMN-major: direction c occupies
 *       P + c*ldp .. P + c*ldp + m - 1 (ldp >= m), in `p_dtype` (EOGP_F16 as
 *       the paper stores it, EOGP_BF16 or EOGP_F32).
 *   X   [N, ldx] fp32, ldx >= k.
 *   ws  eogp_pca_project_workspace_size(N, ...) bytes: the split copy of an
 *       fp32 P, then scratch that lets small batches split the m-long sums
 *       across workgroups (partial sums are added in a fixed order, so the
 *       result does not depend on the split). For EOGP_F16 / EOGP_BF16 P the
 *       workspace may be NULL (no split; slower for small N).
 * With p_dtype EOGP_F16 the fp32 Z is converted to fp16 (split into two fp16
 * parts under EOGP_PREC_ACCURATE); Z must then lie within the fp16 range.
 * ------------------------------------------------------------------------ */
size_t eogp_pca_project_workspace_size(int64_t N, int64_t m, int64_t k, eogp_dtype p_dtype,
                                       eogp_prec prec);
eogp_status eogp_pca_project(const void* Z, eogp_dtype z_dtype, int64_t ldz, int64_t N,
                             int64_t m, const void* P, eogp_dtype p_dtype, int64_t ldp,
                             int64_t k, float* X, int64_t ldx, eogp_prec prec, void* ws,
                             size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * One-bit encoding (eq. onebit; Algorithm 1, storing block: packed sign bits
 * plus an fp16 scale ||x||_1 / k; payload layout of eq. app_payload):
 *   bit c of row i = (X[i, c] >= 0)  (so -0.0 -> 1, NaN -> 0), stored in byte
 *   c >> 3, bit c & 7 of codes + i*code_row_stride (ceil(k/8) bytes written);
 *   scales[i*scale_stride] = fp16 bits of ||X[i, :k]||_1 / k, summed in fp64 and
 *   rounded once to nearest even (overflow gives +inf).
 * Strides let each module's codes and scale land inside a multi-module row.
 * ------------------------------------------------------------------------ */
eogp_status eogp_sign_pack(const float* X, int64_t ldx, int64_t N, int64_t k,
                           uint8_t* codes, int64_t code_row_stride, uint16_t* scales,
                           int64_t scale_stride, void* stream);

/* Tiled store layout (the same bits and scales, stored for streaming; the
 * paper fixes only the byte packing of one module, eq. app_payload). Rows
 * are grouped in tiles of 32; a row of the store holds S = sum_u k_u / 512
 * steps of 64 bytes (each k_u a multiple of 512, module u owning steps
 * step0_u = sum_{v<u} k_v / 512 ..). The 64 bytes of row r = 32 t + i in
 * step s -- bytes 64 (s - step0_u) .. + 63 of module u's row-major code --
 * form, with the other 31 rows of tile t, the 2 KB block t * S + s; their
 * 16-byte piece p (0..3) sits at block offset (p % 2) * 1024 +
 * ((p / 2) * 32 + i) * 16. A store of N rows takes ceil(N / 32) * S * 2048
 * bytes, 16-byte aligned. eogp_sign_pack_tiled writes rows row0 .. row0+N-1
 * of one module (k = k_u bits at step0); the scale goes to scales[i *
 * scale_stride] exactly as for eogp_sign_pack. Bits and scales are those of
 * eogp_sign_pack. Errors: EOGP_ERR_INVALID unless k is a positive multiple of
 * 512, step0 + k / 512 <= steps_per_row, codes is 16-byte aligned and ldx >= k. */
eogp_status eogp_sign_pack_tiled(const float* X, int64_t ldx, int64_t N, int64_t k, int64_t row0,
                                 uint8_t* codes, int64_t steps_per_row, int64_t step0,
                                 uint16_t* scales, int64_t scale_stride, void* stream);

/* ------------------------------------------------------------------------
 * Scoring (eq. onebit_influence, eq. app_stored_influence; Algorithm 1,
 * query block) with a per-query top-k:
 *   score(q, i) = sum_{u = 0..U-1, ascending} s_{i,u} <y_{q,u}, b_{i,u}>,
 * b in {-1, +1}. Each query module vector y_{q,u} is taken in fixed point:
 * f = 14 - e for max_c |y_c| = mu 2^e (mu in [0.5, 1)), y_int = rint(y 2^f)
 * (nearest even), so <y_int, b> is an exact integer n and each term
 * s * n * 2^-f is exact in fp64; an all-zero y_{q,u} contributes 0. Terms are
 * summed in fp64 in module order. Ranking: score descending, then example
 * index ascending.
 *
 *   codes        [N, code_row_stride] bytes; module u occupies bytes
 *                sum_{v<u} k_v/8 .. + k_u/8 of each row (eogp_sign_pack layout).
 *   scales       [N, U] fp16 bit patterns.
 *   k_per_module HOST [U]; each k_u a positive multiple of 64, at most 2^22.
 *   Y            [Q, ldy] fp32 query coordinates (modules concatenated),
 *                ldy >= sum_u k_u.
 *   out_idx      [Q, topk] int64 example indices; out_score [Q, topk] fp32
 *                (the fp64 score rounded once). If N < topk the tail holds
 *                index -1 and score -inf.
 *   full_scores  [Q, N] fp32, or NULL to skip writing every score.
 *   topk         1..256.
 *   ws           eogp_score_topk_workspace_size(N, Q, U, k_per_module, topk) bytes.
 *                With several modules it includes the exact per-(module,
 *                query, row) integer dots of one 16-query pass, U*16*N*4
 *                bytes (8 when some k_u > 2^16), which a second kernel
 *                turns into fp64 terms summed in module order.
 * Requirements: code_row_stride a multiple of 8 and codes 8-byte aligned;
 * Y finite. k_per_module is read on the host during the call (the module
 * table travels in kernel arguments); the call only enqueues work.
 * ------------------------------------------------------------------------ */
size_t eogp_score_topk_workspace_size(int64_t N, int64_t Q, int32_t U,
                                      const int64_t* k_per_module, int32_t topk);
eogp_status eogp_score_topk(const uint8_t* codes, int64_t code_row_stride,
                            const uint16_t* scales, int64_t N, int32_t U,
                            const int64_t* k_per_module, const float* Y, int64_t ldy,
                            int64_t Q, int32_t topk, int64_t* out_idx, float* out_score,
                            float* full_scores, void* ws, size_t ws_bytes, void* stream);

/* Scoring of a store in the tiled layout (see eogp_sign_pack_tiled): the same
 * scores, ranking and outputs as eogp_score_topk on the row-major store with
 * the same bits. Each wave reads one 2 KB block per step as two contiguous
 * 1 KB loads. Every k_u a positive multiple of 512; codes 16-byte aligned,
 * ceil(N / 32) * (sum_u k_u / 512) * 2048 bytes. Workspace:
 * eogp_score_topk_workspace_size with the same arguments. */
eogp_status eogp_score_topk_tiled(const uint8_t* codes, const uint16_t* scales, int64_t N,
                                  int32_t U, const int64_t* k_per_module, const float* Y,
                                  int64_t ldy, int64_t Q, int32_t topk, int64_t* out_idx,
                                  float* out_score, float* full_scores, void* ws,
                                  size_t ws_bytes, void* stream);

/* Scoring without a caller workspace, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid allocation): the same computation, arguments and results as
 * eogp_score_topk, with the workspace taken from a 128 MiB array that the
 * library holds in each GPU's memory until the process ends. The call
 * allocates nothing (no hipMalloc, hipFree or allocating library routine) and
 * only enqueues work on `stream`. Limit: the call's workspace size, as
 * eogp_score_topk_workspace_size reports it, must be at most 128 MiB
 * (134217728 bytes), else EOGP_ERR_INVALID with nothing enqueued. One
 * module of 16,384 bits fits any number of stored rows with up to 3,936
 * queries per call; several modules need 64 bytes per stored row and
 * module for each 16 queries (48 modules of 8,192 bits: about 38,000 rows for
 * 16 queries). All calls on one GPU share that
 * GPU's array: calls that overlap on one GPU (several streams or threads)
 * race and must be serialised by the caller. Other errors as for
 * eogp_score_topk. */
eogp_status eogp_score_topk_noalloc(const uint8_t* codes, int64_t code_row_stride,
                                    const uint16_t* scales, int64_t N, int32_t U,
                                    const int64_t* k_per_module, const float* Y, int64_t ldy,
                                    int64_t Q, int32_t topk, int64_t* out_idx, float* out_score,
                                    float* full_scores, void* stream);

/* ------------------------------------------------------------------------
 * EK-FAC corrected eigenvalues, the fitting pass that precedes selection
 * (Section 2.2, eq. ekfac_eigendecompose: Lambda[j, k] is the mean over
 * examples of the squared coordinate (Q_S^T G_i Q_A)[j, k] of each
 * sequence-level gradient G_i = sum_{valid t} ds_t a_t^T; Appendix C.2).
 * For the batch given, sq_sum[j, k] receives (accumulate = 0) or is
 * incremented by (accumulate != 0) the sum over its N examples of that
 * square; after all batches the caller divides by the total number of
 * examples. Inputs, strides, mask, dtypes and precision modes are those of
 * eogp_rotate_retain.
 *
 *   Q_A, Q_S  [d_in, d_in] and [d_out, d_out] fp32 K-FAC eigenbases.
 *   e_acts, e_grads  power-of-two input scaling of the fp16 mode, as set by
 *             eogp_plan_set_input_exponents for the first stage (in
 *             [-60, 60]; ignored by the other modes). In the fp16 mode the
 *             rotated tokens are also kept in fp16 (relative error of
 *             sq_sum about 1e-3) and the squares are fp16 MFMA products.
 *   sq_sum    [d_out, d_in] fp32, row-major (the layout of eigvals).
 *   ws        at least eogp_ekfac_workspace_size bytes.
 * Errors as for eogp_rotate_retain; EOGP_ERR_INVALID for an exponent outside
 * [-60, 60]. The sum over examples is formed in a fixed order, so repeated
 * calls give identical results.
 * ------------------------------------------------------------------------ */
size_t eogp_ekfac_workspace_size(int64_t N, int64_t T, int64_t d_in, int64_t d_out);
eogp_status eogp_ekfac_eigenvalues(const void* acts, int64_t ld_acts, const void* out_grads,
                                   int64_t ld_grads, eogp_dtype in_dtype,
                                   const uint8_t* token_mask, int64_t N, int64_t T,
                                   int64_t d_in, int64_t d_out, const float* Q_A,
                                   const float* Q_S, eogp_prec prec, int32_t e_acts,
                                   int32_t e_grads, float* sq_sum, int32_t accumulate, void* ws,
                                   size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * PCA fit (appendix on PCA fitting; Proposition rayleigh_ritz): the shared
 * projection P of one module from cached first-stage coordinates Z [n, m],
 * uncentered. The columns of P are the top-k right singular vectors of Z,
 * i.e. the eigenvectors of Z^T Z / n with the largest eigenvalues, recovered
 * from the n x n Gram matrix: Z Z^T v_c = lambda_c v_c (descending),
 * p_c = Z^T v_c / sqrt(lambda_c), mu_c = lambda_c / n.
 *
 *   Z    [n, ldz] fp32, ldz >= m (device).
 *   Pt   [k, ldp] fp32, ldp >= m: row c = p_c, the layout eogp_pca_project
 *        takes; each row is signed so that its largest-magnitude entry (the
 *        first such on ties) is positive; columns m..ldp-1 are not written.
 *   mu   [k] fp32: the eigenvalues of Z^T Z / n, descending.
 * The Gram matrix and Z^T V are formed in fp64 (exact products of the fp32
 * inputs); the symmetric eigendecomposition is rocSOLVER's dsyevdx in the
 * caller's workspace. Cost: 2 n^2 m + 2 n m k flops plus the eigensolver.
 * Errors: EOGP_ERR_INVALID for bad sizes or NULL pointers (need
 * 1 <= k <= min(n, m), n < 2^31) or when Z has fewer than k nonzero
 * singular values (eigenvalues at or below 1e-12 of the largest count as
 * zero); EOGP_ERR_DEVICE if the eigensolver fails; on an error Pt and mu
 * hold unspecified values;
 * EOGP_ERR_WORKSPACE if ws is too small. Synchronises `stream` (the
 * eigensolver's status is read back). The workspace size query needs a GPU
 * (it asks rocSOLVER) and returns 0 if none is usable.
 * ------------------------------------------------------------------------ */
size_t eogp_pca_fit_workspace_size(int64_t n, int64_t m, int64_t k);
eogp_status eogp_pca_fit(const float* Z, int64_t ldz, int64_t n, int64_t m, int64_t k,
                         float* Pt, int64_t ldp, float* mu, void* ws, size_t ws_bytes,
                         void* stream);

/* ------------------------------------------------------------------------
 * Random second stage, EOGP-R (Appendix B.2, eq. app_srht_definition): the
 * subsampled randomized Hadamard transform x = sqrt(p/k) R H_p D J z in place
 * of the PCA projection, for every row z of Z:
 *   J zero-pads the m coordinates to p = 2^ceil(log2 m), D multiplies them by
 *   the random signs, H_p is the orthonormal Walsh-Hadamard matrix in
 *   Sylvester order (entry (r, i) = (-1)^popcount(r & i) / sqrt(p)), and R
 *   keeps rows `rows[0..k)` in that order.
 * The random draws are the caller's (the same realised transform serves the
 * store and the queries).
 *
 *   Z      [N, ldz] fp32, ldz >= m.
 *   signs  [m] int8: negative = -1, otherwise +1.
 *   rows   [k] int32 in [0, p); a row outside gives NaN in that output
 *          column; repeated rows repeat the coordinate.
 *   X      [N, ldx] fp32, ldx >= k; columns k..ldx-1 are not written.
 * Errors: EOGP_ERR_INVALID for bad sizes or NULL pointers, k > p, or
 * ldz < m / ldx < k; EOGP_ERR_UNSUPPORTED for p > 2^20 (m > 1,048,576);
 * EOGP_ERR_WORKSPACE if ws is too small.
 * p <= 32768 needs no workspace (ws may be NULL); larger p are transformed in
 * two stages through ws (eogp_srht_project_workspace_size bytes: one padded
 * fp32 row per example). Enqueued on `stream`.
 * ------------------------------------------------------------------------ */
size_t eogp_srht_project_workspace_size(int64_t N, int64_t m);
eogp_status eogp_srht_project(const float* Z, int64_t ldz, int64_t N, int64_t m,
                              const int8_t* signs, const int32_t* rows, int64_t k, float* X,
                              int64_t ldx, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Kernel timing, for measurement harnesses. While enabled, each launch of a
 * kernel class below is bracketed by two HIP events recorded on the stream it
 * is launched on. eogp_timing_read waits for the recorded events of one class,
 * returns the summed elapsed time and the number of launches, and forgets
 * them. Disabled by default; costs nothing when disabled.
 * ------------------------------------------------------------------------ */
typedef enum {
  EOGP_KT_ROTATION_GEMM = 0,  /* first-stage rotations (two per first-stage call) */
  EOGP_KT_RETAINED = 1,       /* retained products + half-whitening              */
  EOGP_KT_PCA_GEMM = 2,       /* second-stage projection                         */
  EOGP_KT_SIGN_PACK = 3,      /* one-bit encoding                                */
  EOGP_KT_SCORE_PASS = 4,     /* one streaming pass over the codes               */
  EOGP_KT_SCORE_MERGE = 5,    /* top-k merge after a pass                        */
  EOGP_KT_SCORE_PREP = 6,     /* fixed-point query preparation                   */
  EOGP_KT_COMPACTION = 7,     /* valid-token compaction                          */
  EOGP_KT_SRHT = 8,           /* random second stage (EOGP-R)                    */
  EOGP_KT_EKFAC = 9,          /* EK-FAC squared rotated gradients                */
  EOGP_KT_PCA_FIT = 10,       /* PCA fit: Gram and projection contractions       */
  EOGP_KT_COUNT = 11
} eogp_kernel_class;
eogp_status eogp_timing_enable(int32_t enable);
eogp_status eogp_timing_read(int32_t kernel_class, double* total_ms, int64_t* launches);

/* ------------------------------------------------------------------------ */
const char* eogp_status_string(eogp_status status);
const char* eogp_last_error(void);
/* Library version as major*10000 + minor*100 + patch. */
int32_t eogp_version(void);

#ifdef __cplusplus
}
#endif
#endif /* EOGP_H */
