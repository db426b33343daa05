/*
 * loca.h -- C ABI of libloca, the gfx950 (MI355X) implementation of the
 * forward-only per-block adaptation step of LoCA (Local Credit Assignment).
 *
 * After calibration, each outer iteration of the method (Section S13, steps
 * 2-5) needs, for every transformer block l:
 *   (a1) the frozen-head error  E_t = w_t (softmax(z_t) - onehot(y_t))
 *        (Lemma S3.1; Eq. 4);
 *   (a2) the tokenwise feedback through the fixed rank-k credit factors,
 *        Y = E A~ and Q = Y B~ (Sections S3, S11), and the scale-normalised
 *        displacement T = -eta_bar_m Q of each mini-batch m (Eq. 10, S8);
 *   (a3) the streaming Gram S += X_m^T X_m of the block inputs (Eq. 9, S7);
 *   (a4) the streaming cross statistic K += -eta_bar_m X_m^T Y_m, so that the
 *        full cross statistic is Z = X^T T = K B~ (Eq. 9, S7);
 *   (a5) the ridge solve (S + lam I) W = S W_prev + Z by Cholesky
 *        (Eq. 7, Theorem S6.1, S7), and the paper's projected form
 *        B* = C_l (G_l + lam I)^{-1} with a fixed random projection A_l;
 *   (a6) the best rank-r_a approximation of W (Lemma S5.2), returned as
 *        adapter factors A (r_a x d), B (d x r_a) with W_r = A^T B^T.
 *
 * Symbols: X is N x d, one token per row (the block input h_{l-1} at the
 * selected prediction positions); the paper's head W_u^T is folded into the
 * credit factor A~ (C x k), so C is the label-set size (or the vocabulary) and
 * the paper's F_l = U_k S_k V_k^T corresponds to A~ = W_u V_k, B~ = S_k U_k^T.
 *
 * Conventions for every entry point
 *   - All matrices are row-major.  Array pointers are DEVICE pointers owned by
 *     the caller, except `lambdas`, which is a host array.
 *   - Calls are batched over `nb` independent blocks (the Jacobi schedule
 *     solves blocks independently, Section S8).  Per-block arrays of block b
 *     start at base + b * <name>_bstride (in elements of the array's type).
 *   - Work is enqueued on `stream` (a hipStream_t; NULL = the null stream).
 *     The library never synchronises and never allocates device memory.
 *     Scratch memory comes from the caller's `ws`, at least
 *     loca_workspace_size(...) bytes, 256-byte aligned.
 *   - State kept by the library: loca_ridge_solve creates, on its first call
 *     on a device, two internal streams and a few events of that device, and
 *     keeps them until the process ends; creating them and every submission
 *     that uses them run under a per-device mutex.  loca_error_targets_noalloc
 *     uses a fixed device array instead of a workspace (see there).
 *   - Argument errors are detected on the host before anything is enqueued
 *     and returned synchronously (LOCA_E_ARG, LOCA_E_WORKSPACE,
 *     LOCA_E_UNSUPPORTED).  Launch failures return LOCA_E_HIP.  Conditions
 *     found on the device are written to `dev_info` (device int32): 0 when
 *     none, LOCA_INFO_NONFINITE for non-finite data, else the entry point's
 *     own positive code.
 *   - Concurrent calls from several host threads are safe when they use
 *     distinct output, dev_info and workspace buffers (calls of
 *     loca_error_targets_noalloc on one device share its array and must not
 *     overlap).  No C++ exception crosses this interface.
 *   - Precision modes: "bf16 mode" = bf16 X, fp32 statistics (S, K); "fp32
 *     mode" = fp32 X, fp64 statistics.  Other combinations are rejected.
 */
#ifndef LOCA_H
#define LOCA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  LOCA_OK = 0,
  LOCA_E_ARG = 1,          /* invalid argument (null pointer, bad size, stride, lambda <= 0, ...) */
  LOCA_E_WORKSPACE = 2,    /* ws is NULL, misaligned or smaller than loca_workspace_size() */
  LOCA_E_HIP = 3,          /* a HIP launch failed */
  LOCA_E_UNSUPPORTED = 4   /* valid but outside what the library implements (e.g. k > 128) */
} loca_status;

typedef enum { LOCA_F32 = 0, LOCA_BF16 = 1, LOCA_F64 = 2 } loca_dtype;

/* dev_info code of every entry point that checks its data: a non-finite value (NaN, an
 * infinity, or a square that overflows) reached a reduction of the call, whose outputs
 * are then unspecified.  It takes precedence over the positive codes. */
#define LOCA_INFO_NONFINITE (-1)

/* dev_info code of loca_feedback_fit_large: the subspace basis lost rank (a pivot of its
 * Cholesky QR was not positive), so fewer than l directions of the map were found; the
 * outputs are then unspecified. */
#define LOCA_INFO_BASIS_RANK (-2)

typedef enum {
  LOCA_OP_ERROR_TARGETS = 0,
  LOCA_OP_ACCUMULATE_STATS = 1,
  LOCA_OP_RIDGE_SOLVE = 2,
  LOCA_OP_LOWRANK_TRUNCATE = 3,
  LOCA_OP_RIDGE_SOLVE_PROJECTED = 4,
  LOCA_OP_FEEDBACK_FIT = 5,
  LOCA_OP_TOP_ERROR = 6,
  LOCA_OP_CREDIT_FROM_TOP_ERROR = 7,
  LOCA_OP_REALIZATION_ERROR = 8,
  LOCA_OP_CREDIT_GRAM = 9,
  LOCA_OP_FEEDBACK_FIT_PRIMAL = 10,
  LOCA_OP_FEEDBACK_FIT_LARGE = 11,
  LOCA_OP_FUSED_HEAD = 12
} loca_op;

/* Per (block, micro-batch) scalars of the scale-normalised step (Eq. 10).
 * Device-resident, one per block.  RMS ratios use squared Frobenius norms:
 * eta_bar = eta * sqrt(sum_x2 / sum_q2), and eta_bar = 0 when sum_q2 = 0. */
typedef struct {
  double sum_q2;   /* ||Q_m||_F^2, Q_m = Y_m B~ (written by loca_error_targets)      */
  double sum_x2;   /* ||X_m||_F^2 (written by loca_accumulate_stats)                  */
  double eta_bar;  /* absolute step of this micro-batch (written by loca_accumulate_stats) */
  int64_t n;       /* tokens in the micro-batch                                        */
} loca_mb;

typedef void* loca_stream_t; /* hipStream_t */

/* ---------------------------------------------------------------------------
 * (a1, a2) Head error and credit coordinates of one micro-batch.
 *   Lemma S3.1: E_t = w_t (softmax(z_t) - onehot(y_t)) over C classes.
 *   Sections S3, S11: Y = E A~ (n x k) for every block; and
 *   mb[b].sum_q2 = ||Y B~_b||_F^2 = sum_t Y_t (B~ B~^T) Y_t^T, the denominator of
 *   Eq. 10 (the displacement itself is never materialised; see
 *   loca_dense_targets).
 * logits : n x C (ld_logits >= C), F32 or BF16, shared by all blocks.
 * labels : n int32 in [0, C).       w : n float loss weights, or NULL (= 1).
 * a_w : n float statistic weights a_t >= 0 (the weighted statistics of Section S7),
 *       or NULL (= 1); the same array is passed to loca_accumulate_stats.  Then
 *       sum_q2 = sum_t a_t ||Q_t||^2 (the mean squares of Eq. 10 under the weights).
 * credit_a : per block C x k (F32 or BF16), stride a_bstride.
 * credit_b : per block k x d float, stride b_bstride.
 * credit_gram : NULL, or B~ B~^T of every block as written by loca_credit_gram for the same
 *     credit_b (the call then skips forming it; B~ is fixed for a whole step, so the
 *     micro-batches after the first can share one).
 * y_out : per block n x k float, stride y_bstride.
 * e_out : n x C float, or NULL (the error rows, for tests).
 * mb_out : nb entries; sum_q2 and n are written, sum_x2 and eta_bar zeroed.
 * dev_info : one int32; 0, or 1 + the smallest row whose label is out of range
 *            (that row's outputs are then unspecified), or LOCA_INFO_NONFINITE when
 *            ||Q||^2 of some block is not finite (a NaN or +inf logit, or non-finite
 *            weights or credit factors; a -inf logit is an excluded class and is fine).
 * Limits: k <= 128.  Any n >= 1, C >= 1, d >= 1.
 * ------------------------------------------------------------------------- */
loca_status loca_error_targets(loca_stream_t stream, int64_t nb, int64_t n, int64_t C, int64_t k,
                               int64_t d, const void* logits, loca_dtype logits_dtype,
                               int64_t ld_logits, const int32_t* labels, const float* w,
                               const float* a_w, const void* credit_a, loca_dtype a_dtype,
                               int64_t a_bstride,
                               const float* credit_b, int64_t b_bstride, const double* credit_gram,
                               float* y_out, int64_t y_bstride, float* e_out, loca_mb* mb_out,
                               int32_t* dev_info, void* ws, size_t ws_bytes);

/* ---------------------------------------------------------------------------
 * The credit Gram B~_b B~_b^T (k x k, fp64) of every block, the matrix through which
 * loca_error_targets forms ||Q||^2 = sum_t Y_t (B~ B~^T) Y_t^T (Eq. 10's denominator), for
 * callers that form it once per step and pass it to every micro-batch's call.
 * g_out : per block ld x ld doubles, ld = loca_credit_gram_ld(k) (entries past k are zero).
 * Workspace: LOCA_OP_CREDIT_GRAM with nb, d and k.  Limits: k <= 128.
 * ------------------------------------------------------------------------- */
loca_status loca_credit_gram(loca_stream_t stream, int64_t nb, int64_t k, int64_t d, const float* credit_b,
                             int64_t b_bstride, double* g_out, void* ws, size_t ws_bytes);
int64_t loca_credit_gram_ld(int64_t k);

/* ---------------------------------------------------------------------------
 * loca_error_targets without a workspace, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc).  Same arguments, kernels, outputs and dev_info codes as
 * loca_error_targets, minus `ws` and `ws_bytes`: the scratch is a fixed array of
 * loca_error_targets_noalloc_max_bytes() bytes (16 MiB) in the library's device
 * memory, one copy per device, held until the process ends.  The call allocates
 * nothing.  Sizes whose workspace (loca_workspace_size(LOCA_OP_ERROR_TARGETS, ...))
 * exceeds the array return LOCA_E_UNSUPPORTED before anything is enqueued; every
 * small label set up to nb = 48 blocks, n = 65536 tokens and k = 64 fits.
 * Every call on a device uses the same array: calls that overlap on one device (two
 * streams, or two host threads) race and must be serialised by the caller.  The first
 * call on a device looks up the array's address there (LOCA_E_HIP if that fails).
 * ------------------------------------------------------------------------- */
loca_status loca_error_targets_noalloc(loca_stream_t stream, int64_t nb, int64_t n, int64_t C, int64_t k,
                                       int64_t d, const void* logits, loca_dtype logits_dtype,
                                       int64_t ld_logits, const int32_t* labels, const float* w,
                                       const float* a_w, const void* credit_a, loca_dtype a_dtype,
                                       int64_t a_bstride, const float* credit_b, int64_t b_bstride,
                                       const double* credit_gram, float* y_out, int64_t y_bstride,
                                       float* e_out, loca_mb* mb_out, int32_t* dev_info);
size_t loca_error_targets_noalloc_max_bytes(void);

/* ---------------------------------------------------------------------------
 * (a3, a4) Streaming statistics of one micro-batch (Eq. 9; Section S7):
 *   S_b += X_b^T diag(a) X_b        (d x d; the upper triangle j >= i is
 *                                    maintained, entries below it are
 *                                    unspecified and never read),
 *   mb[b].sum_x2 = sum_t a_t ||x_t||^2,  mb[b].eta_bar = eta sqrt(sum_x2/sum_q2) (Eq. 10),
 *   K_b += -eta_bar X_b^T diag(a) Y_b   (d x k),
 * with the statistic weights a (Section S7's weighted form; a = 1 when a_w is NULL).
 * overwrite != 0 (the first micro-batch of a step): S = X_b^T diag(a) X_b and
 * K = -eta_bar X_b^T diag(a) Y_b instead, the old contents of S and K never read (no
 * clearing pass needed); overwrite == 0: the caller has zeroed S and K, or an earlier
 * call of the step has written them.  Each mini-batch uses its own eta_bar (Section S8).
 * x : per block n x d, ldx >= d, x_bstride; BF16 (then acc = F32) or F32
 *     (then acc = F64).  BF16 requires ldx % 8 == 0 and a 16-byte aligned
 *     base; F32 requires ldx % 4 == 0 and 16-byte alignment.
 * y : per block n x k float (from loca_error_targets), y_bstride.
 * a_w : n float weights a_t >= 0 shared by the blocks, or NULL; it must be the
 *       array given to loca_error_targets for this micro-batch.  In bf16 mode each
 *       product a_t x_tj enters the matrix cores as two bf16 parts (about 16
 *       significant bits), at twice the matrix-core work of the unweighted call.
 * mb : in: sum_q2; out: sum_x2, eta_bar, n.   eta >= 0.
 * S, K : per block, type `acc`, strides s_bstride, k_bstride.
 * dev_info : nb int32 or NULL; per block 0, or LOCA_INFO_NONFINITE when ||X_m||^2 or
 *            ||Q_m||^2 is not finite (a NaN or infinite entry of X_m, an entry whose
 *            square overflows, or a non-finite head call); that block's S, K and
 *            eta_bar are then unspecified.
 * Limits: k <= 128.
 * ------------------------------------------------------------------------- */
loca_status loca_accumulate_stats(loca_stream_t stream, int64_t nb, int64_t n, int64_t d, int64_t k,
                                  const void* x, loca_dtype x_dtype, int64_t ldx, int64_t x_bstride,
                                  const float* y, int64_t y_bstride, const float* a_w,
                                  double eta, loca_mb* mb,
                                  void* S, void* K, loca_dtype acc, int64_t s_bstride,
                                  int64_t k_bstride, int overwrite, int32_t* dev_info, void* ws,
                                  size_t ws_bytes);

/* ---------------------------------------------------------------------------
 * (a5) Ridge solve in factored form (Eq. 7; Theorem S6.1; Section S7's
 * positive-definite solve without an explicit inverse).  For block b and each
 * lam_l > 0 (host array `lambdas`, n_lambda entries):
 *   M_{b,l} = (S_b + lam_l I)^{-1} [ S_b Lp_b | K_b ]         (d x (r_prev + k))
 * so that the full-width solution of (S + lam I) W = S W_prev + Z, with the
 * current adapter W_prev = Lp Rp (token-major, d x d, rank r_prev) and
 * Z = K B~, is W = M [Rp; B~].  r_prev = 0 (lp = NULL) is the frozen model.
 * Cholesky of the Jacobi-equilibrated matrix, in fp32 (acc = F32) or fp64
 * (acc = F64).
 * S, K : as produced by loca_accumulate_stats (upper triangle of S read).
 * m_out : float, matrix (b, l) at m_out + (b * n_lambda + l) * m_bstride.
 * w_dense_out : optional float d x d W for matrix (b, l) at
 *               w_dense_out + (b * n_lambda + l) * w_bstride; needs rp and
 *               credit_b (ignored when NULL).
 * dev_info : nb * n_lambda int32; 0, or the 1-based index of a non-positive
 *            pivot (LAPACK potrf convention; a NaN pivot counts as non-positive).
 * Limits: r_prev + k <= 128, n_lambda <= 8, nb * n_lambda <= 65535, d <= 65535.
 * With two or more blocks the blocks are split into up to three groups: the first
 * runs on the caller's stream, the others on two internal streams the library
 * creates on its first call on the device.  The internal streams wait for the
 * caller's stream at entry and the caller's stream waits for them at the end, so
 * the call stays ordered on the caller's stream; calls from several host threads
 * are serialised on the internal streams (see the conventions above).
 * ------------------------------------------------------------------------- */
loca_status loca_ridge_solve(loca_stream_t stream, int64_t nb, int64_t d, int64_t k, const void* S,
                             const void* K, loca_dtype acc, int64_t s_bstride, int64_t k_bstride,
                             const float* lp, const float* rp, int64_t r_prev, int64_t lp_bstride,
                             int64_t rp_bstride, const double* lambdas, int64_t n_lambda,
                             float* m_out, int64_t m_bstride, const float* credit_b,
                             int64_t b_bstride, float* w_dense_out, int64_t w_bstride,
                             int32_t* dev_info, void* ws, size_t ws_bytes);

/* ---------------------------------------------------------------------------
 * (a6) Best rank-r_a approximation (Lemma S5.2, Eckart-Young) of W = M R,
 * M: d x kp, R: kp x d, for nm matrices.  Matrix i reads M at
 * m + i * m_bstride and R at r + (i / r_group) * r_bstride (r_group >= 1 lets
 * several ridge strengths share one B~).  With W = U diag(s) V^T:
 *   a_out = U_{r_a}^T            (r_a x d, orthonormal rows),
 *   b_out = V_{r_a} diag(s_{r_a}) (d x r_a),   so W_{r_a} = a_out^T b_out^T
 * and the adapter acts as h_l = h_bar_l + b_out a_out h_{l-1} (Eq. 1).
 * sigma_out : the kp largest singular values of W, decreasing.
 * Directions of numerically zero singular value (W of rank below r_a, its
 * factors rounded to float: below 1e-6 of the largest singular value, or from
 * the first of two within 1e-5 of it whose squares lie within 1e-10 of the
 * largest square of each other, where the eigensolver cannot separate them;
 * exact zeros on its Jacobi fallback) carry no weight: their b_out columns are
 * zero and their a_out rows an orthonormal completion of the other rows (by
 * Householder reconstruction), so a_out always has orthonormal rows.
 * w_dense_out : optional d x d W_{r_a} (float), stride w_bstride.
 * dev_info : nm int32, 0 (reserved for future conditions).
 * Limits: kp <= 128, r_a <= kp, r_a <= 64, kp <= d.
 * ------------------------------------------------------------------------- */
loca_status loca_lowrank_truncate(loca_stream_t stream, int64_t nm, int64_t d, int64_t kp,
                                  int64_t r_a, const float* m, int64_t m_bstride, const float* r,
                                  int64_t r_bstride, int64_t r_group, float* a_out,
                                  int64_t a_bstride, float* b_out, int64_t b_bstride,
                                  float* sigma_out, int64_t sigma_bstride, float* w_dense_out,
                                  int64_t w_bstride, int32_t* dev_info, void* ws, size_t ws_bytes);

/* ---------------------------------------------------------------------------
 * (a5, paper-literal form) Projected block fit of Eqs. 6-9 with the fixed
 * random projection A_l (r_a x d) of Eq. 1, computed from the full-width
 * statistics:  G_l = A_l S A_l^T,  C_l = B_cur G_l + B~^T K^T A_l^T,
 *              B*_l = C_l (G_l + lam I)^{-1}            (d x r_a)
 * (with features p = A_l x and residual target rho = B_cur p + T_t these are
 * exactly the sums of Eq. 9).  b_cur (d x r_a) may be NULL (frozen model).
 * b_out : float, matrix (b, l) at b_out + (b * n_lambda + l) * bo_bstride.
 * g_out : optional float r_a x r_a G_l per block (stride r_a * r_a).
 * dev_info : nb * n_lambda int32 (non-positive pivot, 1-based).
 * Limits: r_a <= 64, k <= 128, n_lambda <= 8.
 * ------------------------------------------------------------------------- */
loca_status loca_ridge_solve_projected(loca_stream_t stream, int64_t nb, int64_t d, int64_t k,
                                       int64_t r_a, const void* S, const void* K, loca_dtype acc,
                                       int64_t s_bstride, int64_t k_bstride,
                                       const float* credit_b, int64_t b_bstride,
                                       const float* proj_a, int64_t pa_bstride,
                                       const float* b_cur, int64_t bc_bstride,
                                       const double* lambdas, int64_t n_lambda, float* b_out,
                                       int64_t bo_bstride, float* g_out, int32_t* dev_info,
                                       void* ws, size_t ws_bytes);

/* ---------------------------------------------------------------------------
 * Realisation error of the fitted adapters (Section S6): the fit realises the
 * displacement X (W - W_prev) instead of the desired T (all micro-batches stacked), and
 *   E_fit = X (W - W_prev) - T          (the data residual B* P - R of the paper).
 * From the solve's outputs and the statistics, for block b and each lam_l (host array):
 *   out[3 i + 0] = sum_n a_n ||E_fit,n||^2,  out[3 i + 1] = ||T||^2 = sum_m eta_bar_m^2 ||Q_m||^2,
 *   out[3 i + 2] = ||W||_F^2,                i = b * n_lambda + l,
 * so that the ridge objective of Theorem S6.1 is out[0] + lam out[2].  Since (S + lam I) W
 * = S W_prev + Z (Z = K B~), X^T X (W - W_prev) = Z - lam W, and
 *   ||E_fit||^2 = ||T||^2 - tr((W - W_prev)^T Z) - lam tr((W - W_prev)^T W),
 * which needs only k x k products of the factors; the value is exact for the computed M up to
 * the solve's residual, and loses relative accuracy when ||E_fit||^2 << ||T||^2.
 * m : per (b, l) d x kp float (kp = r_prev + k), from loca_ridge_solve: matrix (b, l) at
 *     m + (b * n_lambda + l) * m_bstride.   r : per block kp x d float, [Rp; B~] (r_bstride).
 * K : per block d x k, type acc (r_prev = 0: B~ = r).   lp : per block d x r_prev, or NULL.
 * mb_log : n_mb x nb records of the step's micro-batches, (m, b) at mb_log[m * nb + b].
 * Limits: kp <= 64, n_lambda <= 8.  Workspace: LOCA_OP_REALIZATION_ERROR with nb, d, k,
 * r_a = r_prev and n_lambda.
 * ------------------------------------------------------------------------- */
loca_status loca_realization_error(loca_stream_t stream, int64_t nb, int64_t d, int64_t k, int64_t r_prev,
                                   const float* m, int64_t m_bstride, const float* r, int64_t r_bstride,
                                   const void* K, loca_dtype acc, int64_t k_bstride, const float* lp,
                                   int64_t lp_bstride, const loca_mb* mb_log, int64_t n_mb,
                                   const double* lambdas, int64_t n_lambda, double* out, void* ws,
                                   size_t ws_bytes);

/* ---------------------------------------------------------------------------
 * Dense displacement T = -eta_bar Y B~ (Eq. 10; Section S8) of one micro-batch,
 * n x d float per block (stride t_bstride), from the credit coordinates and
 * the eta_bar written by loca_accumulate_stats.  Not on the hot path (the
 * statistics never need T); provided for tests and callers that want it.
 * ------------------------------------------------------------------------- */
loca_status loca_dense_targets(loca_stream_t stream, int64_t nb, int64_t n, int64_t k, int64_t d,
                               const float* y, int64_t y_bstride, const loca_mb* mb,
                               const float* credit_b, int64_t b_bstride, float* t_out,
                               int64_t t_bstride);

/* ---------------------------------------------------------------------------
 * Stage I calibration of the feedback map, run once before adaptation (Section S5,
 * Eq. 5; the theorem on the feedback ridge solution; the rank-truncation lemma).
 * For nb blocks sharing the probe top errors e (d x np float, row-major: column j
 * is probe position j) and with exact block gradients g_b (d x np float, stride
 * g_bstride), the ridge fit in its dual form
 *   F_hat_b = G_b (E^T E + beta I)^{-1} E^T        (a Cholesky solve in np unknowns)
 * its best rank-k approximation F_b = U_k S_k V_k^T and the credit factors of the
 * hot path (W_u^T folded into the first, as loca_error_targets expects):
 *   bt_out : per block k x d float, B~ = S_k U_k^T (stride bt_bstride);
 *   at_out : per block vocab x k float, A~ = W_u V_k (stride at_bstride); needs
 *            wu (vocab x d, F32 or BF16); both may be NULL (then skipped);
 *   vk_out : per block d x k float, V_k itself (stride vk_bstride), the factor of the
 *            paper-order head (loca_credit_from_top_error); may be NULL;
 *   sigma_out : per block np floats, the singular values of F_hat_b, decreasing;
 *   alpha_out : per block the alignment diagnostic <F_b E, G_b> / (||F_b E|| ||G_b||)
 *               (float64).
 * beta > 0 (finite).  dev_info : nb int32, 0 or the 1-based pivot at which
 * E^T E + beta I failed to be positive definite (only for non-finite data).
 * Limits: np <= 64, np <= d, k <= np.  Workspace: LOCA_OP_FEEDBACK_FIT with
 * n = np.
 * ------------------------------------------------------------------------- */
loca_status loca_feedback_fit(loca_stream_t stream, int64_t nb, int64_t d, int64_t np, int64_t k,
                              const float* e, const float* g, int64_t g_bstride, double beta,
                              const void* wu, loca_dtype wu_dtype, int64_t vocab, float* bt_out,
                              int64_t bt_bstride, float* at_out, int64_t at_bstride, float* vk_out,
                              int64_t vk_bstride, float* sigma_out, double* alpha_out,
                              int32_t* dev_info, void* ws, size_t ws_bytes);

/* -------------------------------------------------------------------------
 * The same Stage I calibration through the primal form of the ridge fit
 * (Section S5, the theorem on the feedback ridge solution):
 *   F_hat_b = G_b E^T (E E^T + beta I)^{-1}        (a Cholesky solve in d unknowns)
 * which equals the dual form up to rounding (push-through identity) and serves probe
 * counts beyond the dual form's limit.  E E^T is formed in float64, the solve runs
 * in float64 (np right-hand sides), then every step after R = E^T (E E^T + beta I)^{-1}
 * is the one loca_feedback_fit takes.  Arguments, layouts and outputs are those of
 * loca_feedback_fit.  dev_info : nb int32, each 0 or the 1-based pivot at which
 * E E^T + beta I failed to be positive definite (the one solve serves every block).
 * Limits: np <= 128, np <= d <= 65535, k <= 64, k <= np.  Workspace:
 * LOCA_OP_FEEDBACK_FIT_PRIMAL with n = np (d x d float64 among it).
 * ------------------------------------------------------------------------- */
loca_status loca_feedback_fit_primal(loca_stream_t stream, int64_t nb, int64_t d, int64_t np, int64_t k,
                                     const float* e, const float* g, int64_t g_bstride, double beta,
                                     const void* wu, loca_dtype wu_dtype, int64_t vocab, float* bt_out,
                                     int64_t bt_bstride, float* at_out, int64_t at_bstride, float* vk_out,
                                     int64_t vk_bstride, float* sigma_out, double* alpha_out,
                                     int32_t* dev_info, void* ws, size_t ws_bytes);

/* -------------------------------------------------------------------------
 * Stage I calibration for any probe count, in particular np > d, where the fitted map
 * F_hat_b = G_b E^T (E E^T + beta I)^{-1} (Section S5, Eq. 5 and the theorem on the feedback
 * ridge solution, primal form) is a full-rank d x d matrix.  R^T = (E E^T + beta I)^{-1} E
 * is solved once (float64 Cholesky, shared by the blocks); the best rank-k approximation
 * of F_hat_b = G_b R (the rank-truncation lemma) is then found by randomised subspace
 * iteration, which never forms F_hat_b: from the caller's start block omega (d x l float,
 * e.g. standard normal, shared by the blocks), q rounds of Y = orth(F_hat Omega),
 * Omega = orth(F_hat^T Y), then Q = orth(F_hat Omega) and the exact rank-k truncation of
 * the Ritz approximation Q Q^T F_hat (orth: Cholesky QR taken twice, float64).  The
 * leading k singular pairs converge at the rate (sigma_{l+1} / sigma_k)^(2q+1) of subspace
 * iteration; q and the oversampled width l are the caller's trade of time for accuracy.
 * Arguments and outputs are those of loca_feedback_fit (e: d x np, g_b: d x np, strides
 * as there), except:
 *   sigma_out : per block l floats (stride l), the Ritz values, decreasing; the leading
 *               k approximate the singular values of F_hat_b;
 *   dev_info : nb int32; 0, the 1-based pivot at which E E^T + beta I failed to be positive
 *              definite (any block), or LOCA_INFO_BASIS_RANK for that block.
 * Limits: k <= l <= 128, l <= d <= 65535, k <= 64, q <= 64, np <= 2^21, nb d l <= 2^31.  Workspace:
 * LOCA_OP_FEEDBACK_FIT_LARGE with n = np and r_a = l (d x d and d x np among it).
 * ------------------------------------------------------------------------- */
loca_status loca_feedback_fit_large(loca_stream_t stream, int64_t nb, int64_t d, int64_t np, int64_t k,
                                    int64_t l, int64_t q, const float* e, const float* g, int64_t g_bstride,
                                    const float* omega, double beta, const void* wu, loca_dtype wu_dtype,
                                    int64_t vocab, float* bt_out, int64_t bt_bstride, float* at_out,
                                    int64_t at_bstride, float* vk_out, int64_t vk_bstride, float* sigma_out,
                                    double* alpha_out, int32_t* dev_info, void* ws, size_t ws_bytes);

/* ---------------------------------------------------------------------------
 * The head in the paper's order (Section S11; the error term of the target equation
 * with Lemma S3.1's head error): the top-layer error at the hidden width, computed
 * once and shared by all blocks,
 *   e_t = W_u^T E_t,   E_t = w_t (softmax(z_t) - onehot(y_t))        (e: n x d),
 * after which each block needs only V_k^T e_t (loca_credit_from_top_error) instead
 * of the folded factor A~ = W_u V_k (loca_error_targets).  The work is 4 n V d
 * matrix-core flops once (the softmax weights enter as two bf16 parts) instead of
 * 2 n V k per block, so it pays when L k > d.
 * logits : n x V (ld_logits >= V), F32 or BF16, 16-byte aligned, ld_logits a multiple
 *          of 8 (BF16) or 4 (F32).   labels : n int32 in [0, V).   w : n floats or NULL.
 * wu : V x d, BF16 only (LOCA_E_UNSUPPORTED otherwise), 16-byte aligned.
 * e_out : n x d float, row stride ld_e >= d.
 * dev_info : one int32; 0, or 1 + the smallest row whose label is out of range.
 * Limits: d % 8 == 0 (LOCA_E_UNSUPPORTED otherwise).  Workspace: LOCA_OP_TOP_ERROR with
 * n, d and C = V.
 * ------------------------------------------------------------------------- */
loca_status loca_top_error(loca_stream_t stream, int64_t n, int64_t V, int64_t d, const void* logits,
                           loca_dtype logits_dtype, int64_t ld_logits, const int32_t* labels,
                           const float* w, const void* wu, loca_dtype wu_dtype, float* e_out,
                           int64_t ld_e, int32_t* dev_info, void* ws, size_t ws_bytes);

/* ---------------------------------------------------------------------------
 * Per block, the credit coordinates of the paper-order head (Section S11,
 * F e = U_k (S_k (V_k^T e))):  Y_b = e V_k,b  (n x k; row t holds V_k^T e_t), and
 *   mb_out[b].sum_q2 = sum_t a_t ||Y_t B~_b||^2   (B~ = S_k U_k^T),
 * the same outputs as loca_error_targets, so loca_accumulate_stats follows as usual.
 * e : n x d float (row stride ld_e), from loca_top_error.
 * credit_v : per block d x k float (stride v_bstride), V_k.
 * credit_b : per block k x d float (stride b_bstride).   a_w : n floats or NULL.
 * y_out : per block n x k float (stride y_bstride).   mb_out : nb entries.
 * Limits: k <= 128.  Workspace: LOCA_OP_CREDIT_FROM_TOP_ERROR with nb, n and k.
 * ------------------------------------------------------------------------- */
loca_status loca_credit_from_top_error(loca_stream_t stream, int64_t nb, int64_t n, int64_t d,
                                       int64_t k, const float* e, int64_t ld_e,
                                       const float* credit_v, int64_t v_bstride,
                                       const float* credit_b, int64_t b_bstride, const float* a_w,
                                       float* y_out, int64_t y_bstride, loca_mb* mb_out, void* ws,
                                       size_t ws_bytes);

/* ---------------------------------------------------------------------------
 * Fused LM head ("Local Targets", Eq. 4, with Lemma S3.1's head error; the head applied
 * once per top error, Section S11): from the final hidden states instead of stored logits,
 *   out_t = w_t ( sum_v softmax(z_t)_v Vm[v, :] - Vm[y_t, :] ),   z_t = W_u h_t,
 * i.e. out = E Vm with E_t = w_t (softmax(z_t) - onehot(y_t)).  The logits are formed on the
 * matrix cores tile by tile (bf16 operands, fp32 accumulation) under an online softmax and
 * never stored; P is applied as bf16 hi + lo parts (about 16 significant bits); the
 * vocabulary ranges are combined in a fixed order in float64.
 *   Vm = W_u       -> out = e, the top error of the paper's order (loca_top_error's output,
 *                     for loca_credit_from_top_error);
 *   Vm = [A~_1 | ... | A~_L] (bf16) -> out = [Y_1 | ... | Y_L], every block's coordinates.
 * h : n x d bf16, row stride ldh (ldh % 8 == 0, 16-byte aligned base).
 * wu : V x d bf16, rows packed (row stride d), 16-byte aligned.
 * labels : n int32 in [0, V).  w : n float loss weights, or NULL (= 1).
 * vm : V x c bf16, row stride ld_vm >= c.   out : n x c float, row stride ld_out >= c.
 * dev_info : one int32: 0, or 1 + the smallest row whose label is out of range (that
 *            row's label term is dropped), or LOCA_INFO_NONFINITE when a token's softmax
 *            sum is not finite (non-finite h or W_u), which takes precedence.
 * Cost: ceil(c / 64) passes of the logits product (the folded order with k <= 64 takes
 * one; the paper's order, c = d, takes d / 64: it trades logits storage for recomputation).
 * Limits: d % 8 == 0 (LOCA_E_UNSUPPORTED otherwise), c <= 2^24, V, d, ldh <= 2^23.
 * Workspace: LOCA_OP_FUSED_HEAD with n, C = V and k = c.
 * ------------------------------------------------------------------------- */
loca_status loca_fused_head(loca_stream_t stream, int64_t n, int64_t V, int64_t d, int64_t c, const void* h,
                            int64_t ldh, const void* wu, const int32_t* labels, const float* w,
                            const void* vm, int64_t ld_vm, float* out, int64_t ld_out, int32_t* dev_info,
                            void* ws, size_t ws_bytes);

/* Workspace bytes for an entry point with the given sizes (nb = blocks, or nm
 * matrices for LOCA_OP_LOWRANK_TRUNCATE; k = kp there; n = np for
 * LOCA_OP_FEEDBACK_FIT and LOCA_OP_FEEDBACK_FIT_PRIMAL, n = np and r_a = l for
 * LOCA_OP_FEEDBACK_FIT_LARGE; C = V and k = c for LOCA_OP_FUSED_HEAD; C = V for LOCA_OP_TOP_ERROR; r_a = r_prev for
 * LOCA_OP_REALIZATION_ERROR).  `acc` selects the precision mode.  Unused arguments
 * may be 0. */
size_t loca_workspace_size(loca_op op, int64_t nb, int64_t n, int64_t d, int64_t k, int64_t C,
                           int64_t r_a, int64_t n_lambda, loca_dtype acc);

const char* loca_status_str(loca_status s);
const char* loca_version(void);

#ifdef __cplusplus
}
#endif

#endif /* LOCA_H */
