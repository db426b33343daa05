// loca_api.hip -- the C ABI of libloca: host-side argument validation and dispatch.
// Every check happens before anything is enqueued, so argument errors are
// reported synchronously and can be tested without a GPU.
#include <new>

#include "loca_launch.h"

using namespace loca;

namespace {

constexpr int64_t kMaxK = 128;
constexpr int64_t kMaxKpTrunc = 128;
constexpr int64_t kMaxRankTrunc = 64;
constexpr int64_t kMaxLambdas = 8;

bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

loca_status check_ws(void* ws, size_t ws_bytes, size_t need) {
  if (need == 0) return LOCA_OK;
  if (!ws || !aligned(ws, 256) || ws_bytes < need) return LOCA_E_WORKSPACE;
  return LOCA_OK;
}

loca_status from_hip(hipError_t e) { return e == hipSuccess ? LOCA_OK : LOCA_E_HIP; }

bool bad_lambdas(const double* l, int64_t nl) {
  if (!l || nl < 1) return true;
  for (int64_t i = 0; i < nl; ++i)
    if (!(l[i] > 0.0) || l[i] == __builtin_inf()) return true;
  return false;
}

}  // namespace

extern "C" {

const char* loca_version(void) { return "libloca 0.1 (gfx950)"; }

const char* loca_status_str(loca_status s) {
  switch (s) {
    case LOCA_OK: return "ok";
    case LOCA_E_ARG: return "invalid argument";
    case LOCA_E_WORKSPACE: return "workspace missing, misaligned or too small";
    case LOCA_E_HIP: return "HIP launch failed";
    case LOCA_E_UNSUPPORTED: return "unsupported size or mode";
  }
  return "unknown status";
}

size_t loca_workspace_size(loca_op op, int64_t nb, int64_t n, int64_t d, int64_t k, int64_t C, int64_t r_a,
                           int64_t n_lambda, loca_dtype acc) {
  if (nb < 1 || k < 1) return 0;
  switch (op) {
    case LOCA_OP_ERROR_TARGETS: return n < 1 ? 0 : error_targets_ws(nb, n, C, k);
    case LOCA_OP_ACCUMULATE_STATS: return d < 1 ? 0 : accumulate_stats_ws(nb, n, d, k, acc);
    case LOCA_OP_RIDGE_SOLVE: return d < 1 || n_lambda < 1 ? 0 : ridge_solve_ws(nb, d, k, n_lambda, acc);
    case LOCA_OP_LOWRANK_TRUNCATE: return lowrank_truncate_ws(nb, d, k, r_a);
    case LOCA_OP_RIDGE_SOLVE_PROJECTED: return projected_ws(nb, d, k, r_a, n_lambda);
    case LOCA_OP_FEEDBACK_FIT: return d < 1 || n < 1 || n > 64 ? 0 : feedback_fit_ws(nb, d, n, k);
    case LOCA_OP_FEEDBACK_FIT_PRIMAL:
      return d < 1 || n < 1 || n > kMaxKpTrunc ? 0 : feedback_fit_primal_ws(nb, d, n, k);
    case LOCA_OP_FUSED_HEAD: return n < 1 || C < 1 || k < 1 ? 0 : fused_head_ws(n, C, k);
    case LOCA_OP_FEEDBACK_FIT_LARGE:
      return d < 1 || n < 1 || r_a < 1 || r_a > kMaxKpTrunc ? 0 : feedback_fit_large_ws(nb, d, n, k, r_a);
    case LOCA_OP_TOP_ERROR: return n < 1 || d < 1 || C < 1 ? 0 : top_error_ws(n, C, d);
    case LOCA_OP_CREDIT_FROM_TOP_ERROR: return n < 1 ? 0 : credit_from_top_error_ws(nb, n, k);
    case LOCA_OP_CREDIT_GRAM: return d < 1 ? 0 : credit_gram_ws(nb, k);
    case LOCA_OP_REALIZATION_ERROR:
      return d < 1 || n_lambda < 1 || r_a < 0 ? 0 : realization_error_ws(nb, d, k, r_a, n_lambda);
  }
  return 0;
}

static loca_status check_error_args(int64_t nb, int64_t n, int64_t C, int64_t k, int64_t d, const void* logits,
                                    loca_dtype logits_dtype, int64_t ld_logits, const int32_t* labels,
                                    const void* credit_a, loca_dtype a_dtype, int64_t a_bstride, const float* credit_b,
                                    int64_t b_bstride, const float* y_out, int64_t y_bstride, const loca_mb* mb_out,
                                    const int32_t* dev_info) {
  if (nb < 1 || n < 1 || C < 1 || k < 1 || d < 1) return LOCA_E_ARG;
  if (!logits || !labels || !credit_a || !credit_b || !y_out || !mb_out || !dev_info) return LOCA_E_ARG;
  if (ld_logits < C) return LOCA_E_ARG;
  if (logits_dtype != LOCA_F32 && logits_dtype != LOCA_BF16) return LOCA_E_ARG;
  if (a_dtype != LOCA_F32 && a_dtype != LOCA_BF16) return LOCA_E_ARG;
  if (nb > 1 && (a_bstride < C * k || b_bstride < k * d || y_bstride < n * k)) return LOCA_E_ARG;
  if (n > (int64_t)INT32_MAX - 1 || nb > 65535) return LOCA_E_UNSUPPORTED;
  if (k > kMaxK) return LOCA_E_UNSUPPORTED;
  return LOCA_OK;
}

loca_status loca_error_targets(loca_stream_t stream, int64_t nb, int64_t n, int64_t C, int64_t k, int64_t d,
                               const void* logits, loca_dtype logits_dtype, int64_t ld_logits,
                               const int32_t* labels, const float* w, const float* a_w, const void* credit_a,
                               loca_dtype a_dtype,
                               int64_t a_bstride, const float* credit_b, int64_t b_bstride,
                               const double* credit_gram, float* y_out,
                               int64_t y_bstride, float* e_out, loca_mb* mb_out, int32_t* dev_info, void* ws,
                               size_t ws_bytes) {
  loca_status st = check_error_args(nb, n, C, k, d, logits, logits_dtype, ld_logits, labels, credit_a, a_dtype,
                                    a_bstride, credit_b, b_bstride, y_out, y_bstride, mb_out, dev_info);
  if (st != LOCA_OK) return st;
  st = check_ws(ws, ws_bytes, error_targets_ws(nb, n, C, k));
  if (st != LOCA_OK) return st;
  ErrorArgs a{(hipStream_t)stream, nb, n, C, k, d, ld_logits, logits, logits_dtype, labels, w, a_w, credit_a, a_dtype,
              a_bstride, credit_b, b_bstride, credit_gram, y_out, y_bstride, e_out, mb_out, dev_info, (char*)ws};
  return from_hip(launch_error_targets(a));
}

int64_t loca_credit_gram_ld(int64_t k) { return k < 1 ? 0 : credit_gram_ld(k); }

loca_status loca_credit_gram(loca_stream_t stream, int64_t nb, int64_t k, int64_t d, const float* credit_b,
                             int64_t b_bstride, double* g_out, void* ws, size_t ws_bytes) {
  if (nb < 1 || k < 1 || d < 1 || !credit_b || !g_out) return LOCA_E_ARG;
  if (nb > 1 && b_bstride < k * d) return LOCA_E_ARG;
  if (k > kMaxK || nb > 65535) return LOCA_E_UNSUPPORTED;
  loca_status st = check_ws(ws, ws_bytes, credit_gram_ws(nb, k));
  if (st != LOCA_OK) return st;
  return from_hip(launch_credit_gram_only((hipStream_t)stream, nb, k, d, credit_b, b_bstride, g_out, (char*)ws));
}

loca_status loca_error_targets_noalloc(loca_stream_t stream, int64_t nb, int64_t n, int64_t C, int64_t k, int64_t d,
                                       const void* logits, loca_dtype logits_dtype, int64_t ld_logits,
                                       const int32_t* labels, const float* w, const float* a_w,
                                       const void* credit_a, loca_dtype a_dtype, int64_t a_bstride,
                                       const float* credit_b, int64_t b_bstride, const double* credit_gram,
                                       float* y_out, int64_t y_bstride,
                                       float* e_out, loca_mb* mb_out, int32_t* dev_info) {
  loca_status st = check_error_args(nb, n, C, k, d, logits, logits_dtype, ld_logits, labels, credit_a, a_dtype,
                                    a_bstride, credit_b, b_bstride, y_out, y_bstride, mb_out, dev_info);
  if (st != LOCA_OK) return st;
  if (error_targets_ws(nb, n, C, k) > error_targets_scratch_bytes()) return LOCA_E_UNSUPPORTED;
  void* scratch_ptr = nullptr;
  if (error_targets_scratch(&scratch_ptr) != hipSuccess) return LOCA_E_HIP;
  ErrorArgs a{(hipStream_t)stream, nb, n, C, k, d, ld_logits, logits, logits_dtype, labels, w, a_w, credit_a, a_dtype,
              a_bstride, credit_b, b_bstride, credit_gram, y_out, y_bstride, e_out, mb_out, dev_info,
              (char*)scratch_ptr};
  return from_hip(launch_error_targets(a));
}

size_t loca_error_targets_noalloc_max_bytes(void) { return error_targets_scratch_bytes(); }

loca_status loca_accumulate_stats(loca_stream_t stream, int64_t nb, int64_t n, int64_t d, int64_t k, const void* x,
                                  loca_dtype x_dtype, int64_t ldx, int64_t x_bstride, const float* y,
                                  int64_t y_bstride, const float* a_w, double eta, loca_mb* mb, void* S, void* K,
                                  loca_dtype acc,
                                  int64_t s_bstride, int64_t k_bstride, int overwrite, int32_t* dev_info,
                                  void* ws, size_t ws_bytes) {
  if (nb < 1 || n < 1 || d < 1 || k < 1) return LOCA_E_ARG;
  if (!x || !y || !mb || !S || !K) return LOCA_E_ARG;
  if (!(eta >= 0.0) || eta == __builtin_inf()) return LOCA_E_ARG;
  if (ldx < d) return LOCA_E_ARG;
  const bool bf = (x_dtype == LOCA_BF16 && acc == LOCA_F32);
  const bool fp = (x_dtype == LOCA_F32 && acc == LOCA_F64);
  if (!bf && !fp) return LOCA_E_ARG;
  if (bf && (ldx % 8 != 0 || !aligned(x, 16) || (nb > 1 && x_bstride % 8 != 0))) return LOCA_E_ARG;
  if (fp && (ldx % 4 != 0 || !aligned(x, 16) || (nb > 1 && x_bstride % 4 != 0))) return LOCA_E_ARG;
  if (nb > 1 && (x_bstride < n * ldx || y_bstride < n * k || s_bstride < d * d || k_bstride < d * k))
    return LOCA_E_ARG;
  if (k > kMaxK) return LOCA_E_UNSUPPORTED;
  if (nb > 65535 || d > 65535 * 64) return LOCA_E_UNSUPPORTED;
  loca_status st = check_ws(ws, ws_bytes, accumulate_stats_ws(nb, n, d, k, acc));
  if (st != LOCA_OK) return st;
  StatsArgs a{(hipStream_t)stream, nb, n, d, k, x, x_dtype, ldx, x_bstride, y, y_bstride, a_w, eta, mb, S, K, acc,
              s_bstride, k_bstride, dev_info, (char*)ws, overwrite != 0};
  return from_hip(launch_accumulate_stats(a));
}

loca_status loca_ridge_solve(loca_stream_t stream, int64_t nb, int64_t d, int64_t k, const void* S, const void* K,
                             loca_dtype acc, int64_t s_bstride, int64_t k_bstride, const float* lp, const float* rp,
                             int64_t r_prev, int64_t lp_bstride, int64_t rp_bstride, const double* lambdas,
                             int64_t n_lambda, float* m_out, int64_t m_bstride, const float* credit_b,
                             int64_t b_bstride, float* w_dense_out, int64_t w_bstride, int32_t* dev_info, void* ws,
                             size_t ws_bytes) {
  if (nb < 1 || d < 1 || k < 1 || r_prev < 0) return LOCA_E_ARG;
  if (!S || !K || !m_out || !dev_info) return LOCA_E_ARG;
  if (acc != LOCA_F32 && acc != LOCA_F64) return LOCA_E_ARG;
  if (bad_lambdas(lambdas, n_lambda)) return LOCA_E_ARG;
  if (r_prev > 0 && (!lp || (nb > 1 && lp_bstride < d * r_prev))) return LOCA_E_ARG;
  const int64_t m = r_prev + k;
  if (m_bstride < d * m && (nb * n_lambda > 1)) return LOCA_E_ARG;
  if (nb > 1 && (s_bstride < d * d || k_bstride < d * k)) return LOCA_E_ARG;
  if (w_dense_out) {
    if (!credit_b || (nb > 1 && b_bstride < k * d) || (nb * n_lambda > 1 && w_bstride < d * d)) return LOCA_E_ARG;
    if (r_prev > 0) return LOCA_E_UNSUPPORTED;
  }
  (void)rp;
  (void)rp_bstride;
  if (m > kMaxK || n_lambda > kMaxLambdas) return LOCA_E_UNSUPPORTED;
  if (nb * n_lambda > 65535 || d > 65535) return LOCA_E_UNSUPPORTED;
  loca_status st = check_ws(ws, ws_bytes, ridge_solve_ws(nb, d, m, n_lambda, acc));
  if (st != LOCA_OK) return st;
  SolveArgs a{(hipStream_t)stream, nb, d, k, S, K, acc, s_bstride, k_bstride, lp, rp, r_prev, lp_bstride,
              rp_bstride, lambdas, n_lambda, m_out, m_bstride, credit_b, b_bstride, w_dense_out, w_bstride,
              dev_info, (char*)ws};
  return from_hip(launch_ridge_solve(a));
}

loca_status loca_lowrank_truncate(loca_stream_t stream, int64_t nm, int64_t d, int64_t kp, int64_t r_a,
                                  const float* m, int64_t m_bstride, const float* r, int64_t r_bstride,
                                  int64_t r_group, float* a_out, int64_t a_bstride, float* b_out, int64_t b_bstride,
                                  float* sigma_out, int64_t sigma_bstride, float* w_dense_out, int64_t w_bstride,
                                  int32_t* dev_info, void* ws, size_t ws_bytes) {
  if (nm < 1 || d < 1 || kp < 1 || r_a < 1 || r_group < 1) return LOCA_E_ARG;
  if (!m || !r || !a_out || !b_out || !sigma_out || !dev_info) return LOCA_E_ARG;
  if (r_a > kp || kp > d) return LOCA_E_ARG;
  if (nm > 1 && (m_bstride < d * kp || a_bstride < r_a * d || b_bstride < d * r_a || sigma_bstride < kp))
    return LOCA_E_ARG;
  if (nm > r_group && r_bstride < kp * d) return LOCA_E_ARG;
  if (w_dense_out && nm > 1 && w_bstride < d * d) return LOCA_E_ARG;
  if (kp > kMaxKpTrunc || r_a > kMaxRankTrunc) return LOCA_E_UNSUPPORTED;
  if (nm > 65535 || d > 65535) return LOCA_E_UNSUPPORTED;
  loca_status st = check_ws(ws, ws_bytes, lowrank_truncate_ws(nm, d, kp, r_a));
  if (st != LOCA_OK) return st;
  TruncArgs a{(hipStream_t)stream, nm, d, kp, r_a, m, m_bstride, r, r_bstride, r_group, a_out, a_bstride, b_out,
              b_bstride, sigma_out, sigma_bstride, w_dense_out, w_bstride, dev_info, (char*)ws};
  return from_hip(launch_lowrank_truncate(a));
}

loca_status loca_ridge_solve_projected(loca_stream_t stream, int64_t nb, int64_t d, int64_t k, int64_t r_a,
                                       const void* S, const void* K, loca_dtype acc, int64_t s_bstride,
                                       int64_t k_bstride, const float* credit_b, int64_t b_bstride,
                                       const float* proj_a, int64_t pa_bstride, const float* b_cur,
                                       int64_t bc_bstride, const double* lambdas, int64_t n_lambda, float* b_out,
                                       int64_t bo_bstride, float* g_out, int32_t* dev_info, void* ws,
                                       size_t ws_bytes) {
  if (nb < 1 || d < 1 || k < 1 || r_a < 1) return LOCA_E_ARG;
  if (!S || !K || !credit_b || !proj_a || !b_out || !dev_info) return LOCA_E_ARG;
  if (acc != LOCA_F32 && acc != LOCA_F64) return LOCA_E_ARG;
  if (bad_lambdas(lambdas, n_lambda)) return LOCA_E_ARG;
  if (nb > 1 && (s_bstride < d * d || k_bstride < d * k || b_bstride < k * d || pa_bstride < r_a * d ||
                 (b_cur && bc_bstride < d * r_a)))
    return LOCA_E_ARG;
  if (nb * n_lambda > 1 && bo_bstride < d * r_a) return LOCA_E_ARG;
  if (r_a > kMaxRankTrunc || k > kMaxK || n_lambda > kMaxLambdas) return LOCA_E_UNSUPPORTED;
  if (nb * n_lambda > 65535) return LOCA_E_UNSUPPORTED;
  loca_status st = check_ws(ws, ws_bytes, projected_ws(nb, d, k, r_a, n_lambda));
  if (st != LOCA_OK) return st;
  ProjArgs a{(hipStream_t)stream, nb, d, k, r_a, S, K, acc, s_bstride, k_bstride, credit_b, b_bstride, proj_a,
             pa_bstride, b_cur, bc_bstride, lambdas, n_lambda, b_out, bo_bstride, g_out, dev_info, (char*)ws};
  return from_hip(launch_ridge_solve_projected(a));
}

loca_status loca_realization_error(loca_stream_t stream, int64_t nb, int64_t d, int64_t k, int64_t r_prev,
                                   const float* m, int64_t m_bstride, const float* r, int64_t r_bstride,
                                   const void* K, loca_dtype acc, int64_t k_bstride, const float* lp,
                                   int64_t lp_bstride, const loca_mb* mb_log, int64_t n_mb, const double* lambdas,
                                   int64_t n_lambda, double* out, void* ws, size_t ws_bytes) {
  if (nb < 1 || d < 1 || k < 1 || r_prev < 0 || n_mb < 0) return LOCA_E_ARG;
  if (!m || !r || !K || !out || (n_mb > 0 && !mb_log)) return LOCA_E_ARG;
  if (acc != LOCA_F32 && acc != LOCA_F64) return LOCA_E_ARG;
  if (bad_lambdas(lambdas, n_lambda)) return LOCA_E_ARG;
  const int64_t kp = r_prev + k;
  if (r_prev > 0 && (!lp || (nb > 1 && lp_bstride < d * r_prev))) return LOCA_E_ARG;
  if ((nb * n_lambda > 1 && m_bstride < d * kp) || (nb > 1 && (r_bstride < kp * d || k_bstride < d * k)))
    return LOCA_E_ARG;
  if (kp > 64 || n_lambda > kMaxLambdas) return LOCA_E_UNSUPPORTED;
  if (nb > 65535 || nb * n_lambda > 65535) return LOCA_E_UNSUPPORTED;
  loca_status st = check_ws(ws, ws_bytes, realization_error_ws(nb, d, k, r_prev, n_lambda));
  if (st != LOCA_OK) return st;
  FitArgs a{(hipStream_t)stream, nb, d, k, r_prev, m, m_bstride, r, r_bstride, K, acc, k_bstride, lp, lp_bstride,
            mb_log, n_mb, lambdas, n_lambda, out, (char*)ws};
  return from_hip(launch_realization_error(a));
}

loca_status loca_dense_targets(loca_stream_t stream, int64_t nb, int64_t n, int64_t k, int64_t d, const float* y,
                               int64_t y_bstride, const loca_mb* mb, const float* credit_b, int64_t b_bstride,
                               float* t_out, int64_t t_bstride) {
  if (nb < 1 || n < 1 || k < 1 || d < 1) return LOCA_E_ARG;
  if (!y || !mb || !credit_b || !t_out) return LOCA_E_ARG;
  if (nb > 1 && (y_bstride < n * k || b_bstride < k * d || t_bstride < n * d)) return LOCA_E_ARG;
  if (n > 65535 || nb > 65535) return LOCA_E_UNSUPPORTED;
  return from_hip(launch_dense_targets((hipStream_t)stream, nb, n, k, d, y, y_bstride, mb, credit_b, b_bstride,
                                       t_out, t_bstride));
}

namespace {

loca_status feedback_fit(loca_stream_t stream, int64_t nb, int64_t d, int64_t np, int64_t k, const float* e,
                         const float* g, int64_t g_bstride, double beta, const void* wu, loca_dtype wu_dtype,
                         int64_t vocab, float* bt_out, int64_t bt_bstride, float* at_out, int64_t at_bstride,
                         float* vk_out, int64_t vk_bstride, float* sigma_out, double* alpha_out, int32_t* dev_info,
                         void* ws, size_t ws_bytes, bool primal) {
  if (nb < 1 || d < 1 || np < 1 || k < 1) return LOCA_E_ARG;
  if (!e || !g || !bt_out || !sigma_out || !alpha_out || !dev_info) return LOCA_E_ARG;
  if (!(beta > 0.0) || beta == __builtin_inf()) return LOCA_E_ARG;
  if (k > np || k > d) return LOCA_E_ARG;
  if (nb > 1 && (g_bstride < d * np || bt_bstride < k * d)) return LOCA_E_ARG;
  if (np > d) return LOCA_E_UNSUPPORTED;  // the factored truncation takes np <= d columns
  if (at_out && (!wu || vocab < 1 || (wu_dtype != LOCA_F32 && wu_dtype != LOCA_BF16) ||
                 (nb > 1 && at_bstride < vocab * k)))
    return LOCA_E_ARG;
  if (vk_out && nb > 1 && vk_bstride < d * k) return LOCA_E_ARG;
  if (np > (primal ? kMaxKpTrunc : 64)) return LOCA_E_UNSUPPORTED;
  if (primal && (np > kMaxK || k > kMaxRankTrunc || d > 65535)) return LOCA_E_UNSUPPORTED;
  if (nb > 65535 || d > (int64_t)1 << 30 || vocab > (int64_t)1 << 32) return LOCA_E_UNSUPPORTED;
  loca_status st =
      check_ws(ws, ws_bytes, primal ? feedback_fit_primal_ws(nb, d, np, k) : feedback_fit_ws(nb, d, np, k));
  if (st != LOCA_OK) return st;
  CalibArgs a{(hipStream_t)stream, nb, d, np, k, e, g, g_bstride, beta, wu, wu_dtype, vocab, bt_out, bt_bstride,
              at_out, at_bstride, vk_out, vk_bstride, sigma_out, alpha_out, dev_info, (char*)ws, primal};
  return from_hip(launch_feedback_fit(a));
}

}  // namespace

loca_status loca_feedback_fit(loca_stream_t stream, int64_t nb, int64_t d, int64_t np, int64_t k, const float* e,
                              const float* g, int64_t g_bstride, double beta, const void* wu, loca_dtype wu_dtype,
                              int64_t vocab, float* bt_out, int64_t bt_bstride, float* at_out, int64_t at_bstride,
                              float* vk_out, int64_t vk_bstride, float* sigma_out, double* alpha_out,
                              int32_t* dev_info, void* ws, size_t ws_bytes) {
  return feedback_fit(stream, nb, d, np, k, e, g, g_bstride, beta, wu, wu_dtype, vocab, bt_out, bt_bstride, at_out,
                      at_bstride, vk_out, vk_bstride, sigma_out, alpha_out, dev_info, ws, ws_bytes, false);
}

loca_status loca_feedback_fit_primal(loca_stream_t stream, int64_t nb, int64_t d, int64_t np, int64_t k,
                                     const float* e, const float* g, int64_t g_bstride, double beta, const void* wu,
                                     loca_dtype wu_dtype, int64_t vocab, float* bt_out, int64_t bt_bstride,
                                     float* at_out, int64_t at_bstride, float* vk_out, int64_t vk_bstride,
                                     float* sigma_out, double* alpha_out, int32_t* dev_info, void* ws,
                                     size_t ws_bytes) {
  return feedback_fit(stream, nb, d, np, k, e, g, g_bstride, beta, wu, wu_dtype, vocab, bt_out, bt_bstride, at_out,
                      at_bstride, vk_out, vk_bstride, sigma_out, alpha_out, dev_info, ws, ws_bytes, true);
}

loca_status loca_feedback_fit_large(loca_stream_t stream, int64_t nb, int64_t d, int64_t np, int64_t k, int64_t l,
                                    int64_t q, const float* e, const float* g, int64_t g_bstride, const float* omega,
                                    double beta, const void* wu, loca_dtype wu_dtype, int64_t vocab, float* bt_out,
                                    int64_t bt_bstride, float* at_out, int64_t at_bstride, float* vk_out,
                                    int64_t vk_bstride, float* sigma_out, double* alpha_out, int32_t* dev_info,
                                    void* ws, size_t ws_bytes) {
  if (nb < 1 || d < 1 || np < 1 || k < 1 || l < 1 || q < 0) return LOCA_E_ARG;
  if (!e || !g || !omega || !bt_out || !sigma_out || !alpha_out || !dev_info) return LOCA_E_ARG;
  if (!(beta > 0.0) || beta == __builtin_inf()) return LOCA_E_ARG;
  if (k > l || l > d) return LOCA_E_ARG;
  if (nb > 1 && (g_bstride < d * np || bt_bstride < k * d)) return LOCA_E_ARG;
  if (at_out && (!wu || vocab < 1 || (wu_dtype != LOCA_F32 && wu_dtype != LOCA_BF16) ||
                 (nb > 1 && at_bstride < vocab * k)))
    return LOCA_E_ARG;
  if (vk_out && nb > 1 && vk_bstride < d * k) return LOCA_E_ARG;
  if (l > kMaxKpTrunc || k > kMaxRankTrunc || q > 64) return LOCA_E_UNSUPPORTED;
  if (nb > 65535 || d > 65535 || np > ((int64_t)1 << 21) || vocab > (int64_t)1 << 32) return LOCA_E_UNSUPPORTED;
  if (nb * d * l > ((int64_t)1 << 31)) return LOCA_E_UNSUPPORTED;  // one-dimensional element grids
  loca_status st = check_ws(ws, ws_bytes, feedback_fit_large_ws(nb, d, np, k, l));
  if (st != LOCA_OK) return st;
  CalibArgs a{(hipStream_t)stream, nb, d, np, k, e, g, g_bstride, beta, wu, wu_dtype, vocab, bt_out, bt_bstride,
              at_out, at_bstride, vk_out, vk_bstride, sigma_out, alpha_out, dev_info, (char*)ws, true, l, q, omega};
  return from_hip(launch_feedback_fit_large(a));
}

loca_status loca_fused_head(loca_stream_t stream, int64_t n, int64_t V, int64_t d, int64_t c, const void* h,
                            int64_t ldh, const void* wu, const int32_t* labels, const float* w, const void* vm,
                            int64_t ld_vm, float* out, int64_t ld_out, int32_t* dev_info, void* ws,
                            size_t ws_bytes) {
  if (n < 1 || V < 1 || d < 1 || c < 1) return LOCA_E_ARG;
  if (!h || !wu || !labels || !vm || !out || !dev_info) return LOCA_E_ARG;
  if (ldh < d || ld_vm < c || ld_out < c) return LOCA_E_ARG;
  if (!aligned(h, 16) || !aligned(wu, 16) || ldh % 8 != 0) return LOCA_E_ARG;
  if (d % 8 != 0) return LOCA_E_UNSUPPORTED;
  if (n > (int64_t)INT32_MAX - 1 || V > ((int64_t)1 << 23) || c > ((int64_t)1 << 24)) return LOCA_E_UNSUPPORTED;
  if (d > ((int64_t)1 << 23) || ldh > ((int64_t)1 << 23)) return LOCA_E_UNSUPPORTED;  // 32-bit buffer offsets
  if (((n + 127) / 128) * ((c + 63) / 64) * kMaxFusedSplits > (int64_t)INT32_MAX) return LOCA_E_UNSUPPORTED;
  loca_status st = check_ws(ws, ws_bytes, fused_head_ws(n, V, c));
  if (st != LOCA_OK) return st;
  FusedArgs a{(hipStream_t)stream, n, V, d, c, (const uint16_t*)h, ldh, (const uint16_t*)wu, labels, w,
              (const uint16_t*)vm, ld_vm, out, ld_out, dev_info, (char*)ws};
  return from_hip(launch_fused_head(a));
}

loca_status loca_top_error(loca_stream_t stream, int64_t n, int64_t V, int64_t d, const void* logits,
                           loca_dtype logits_dtype, int64_t ld_logits, const int32_t* labels, const float* w,
                           const void* wu, loca_dtype wu_dtype, float* e_out, int64_t ld_e, int32_t* dev_info,
                           void* ws, size_t ws_bytes) {
  if (n < 1 || V < 1 || d < 1) return LOCA_E_ARG;
  if (!logits || !labels || !wu || !e_out || !dev_info) return LOCA_E_ARG;
  if (ld_logits < V || ld_e < d) return LOCA_E_ARG;
  if (logits_dtype != LOCA_F32 && logits_dtype != LOCA_BF16) return LOCA_E_ARG;
  if (wu_dtype != LOCA_F32 && wu_dtype != LOCA_BF16) return LOCA_E_ARG;
  if (!aligned(logits, 16) || !aligned(wu, 16)) return LOCA_E_ARG;
  if (ld_logits % (logits_dtype == LOCA_BF16 ? 8 : 4) != 0) return LOCA_E_ARG;
  if (wu_dtype != LOCA_BF16 || d % 8 != 0) return LOCA_E_UNSUPPORTED;
  if (n > (int64_t)INT32_MAX - 1 || V > (int64_t)INT32_MAX || (n + 127) / 128 > 65535 || (d + 127) / 128 > 65535)
    return LOCA_E_UNSUPPORTED;
  loca_status st = check_ws(ws, ws_bytes, top_error_ws(n, V, d));
  if (st != LOCA_OK) return st;
  TopErrorArgs a{(hipStream_t)stream, n, V, d, logits, logits_dtype, ld_logits, labels, w, wu, e_out, ld_e, dev_info,
                 (char*)ws};
  return from_hip(launch_top_error(a));
}

loca_status loca_credit_from_top_error(loca_stream_t stream, int64_t nb, int64_t n, int64_t d, int64_t k,
                                       const float* e, int64_t ld_e, const float* credit_v, int64_t v_bstride,
                                       const float* credit_b, int64_t b_bstride, const float* a_w, float* y_out,
                                       int64_t y_bstride, loca_mb* mb_out, void* ws, size_t ws_bytes) {
  if (nb < 1 || n < 1 || d < 1 || k < 1) return LOCA_E_ARG;
  if (!e || !credit_v || !credit_b || !y_out || !mb_out) return LOCA_E_ARG;
  if (ld_e < d) return LOCA_E_ARG;
  if (nb > 1 && (v_bstride < d * k || b_bstride < k * d || y_bstride < n * k)) return LOCA_E_ARG;
  if (k > kMaxK) return LOCA_E_UNSUPPORTED;
  if (nb > 65535 || (n + 63) / 64 > (int64_t)INT32_MAX) return LOCA_E_UNSUPPORTED;
  loca_status st = check_ws(ws, ws_bytes, credit_from_top_error_ws(nb, n, k));
  if (st != LOCA_OK) return st;
  CreditArgs a{(hipStream_t)stream, nb, n, d, k, e, ld_e, credit_v, v_bstride, credit_b, b_bstride, a_w, y_out,
               y_bstride, mb_out, (char*)ws};
  return from_hip(launch_credit_from_top_error(a));
}

}  // extern "C"
