// loca_launch.h -- argument records and launchers of the libloca entry points (host side),
// defined in the kernel files and called by loca_api.hip.
#pragma once

#include "loca_common.h"

// Internal launchers (defined in the kernel files, called by loca_api.hip).
namespace loca {
struct ErrorArgs {
  hipStream_t stream;
  int64_t nb, n, C, k, d, ld_logits;
  const void* logits; loca_dtype logits_dtype;
  const int32_t* labels; const float* w; const float* a_w;
  const void* credit_a; loca_dtype a_dtype; int64_t a_bstride;
  const float* credit_b; int64_t b_bstride;
  const double* credit_gram;  // B~ B~^T per block (loca_credit_gram), or null
  float* y_out; int64_t y_bstride;
  float* e_out; loca_mb* mb_out; int32_t* dev_info;
  char* ws;
};
size_t error_targets_ws(int64_t nb, int64_t n, int64_t C, int64_t k);
int64_t credit_gram_ld(int64_t k);
size_t credit_gram_ws(int64_t nb, int64_t k);
hipError_t launch_credit_gram_only(hipStream_t st, int64_t nb, int64_t k, int64_t d, const float* B,
                                   int64_t b_bstride, double* G, char* ws);
hipError_t launch_error_targets(const ErrorArgs& a);
// the fixed scratch array of loca_error_targets_noalloc: its size, and its address on the
// current device (looked up on the first call on that device)
size_t error_targets_scratch_bytes();
hipError_t error_targets_scratch(void** out);

// The head in the paper's order (Section S11): e = W_u^T E once, then V_k^T e per block.
struct TopErrorArgs {
  hipStream_t stream;
  int64_t n, V, d;
  const void* logits; loca_dtype logits_dtype; int64_t ld_logits;
  const int32_t* labels; const float* w;
  const void* wu;
  float* e_out; int64_t ld_e;
  int32_t* dev_info;
  char* ws;
};
size_t top_error_ws(int64_t n, int64_t V, int64_t d);
hipError_t launch_top_error(const TopErrorArgs& a);

// out_g = w (softmax(z) - onehot(y)) W_g for `groups` right operands W_g (V x kc bf16, stride
// w_bstride), one matrix-core product over the vocabulary; the softmax statistics go to the
// workspace, bad labels to dev_info (atomicMin of 1 + row; the caller initialises it).
struct SoftmaxProductArgs {
  hipStream_t stream;
  int64_t n, V;
  const void* logits; loca_dtype logits_dtype; int64_t ld_logits;
  const int32_t* labels; const float* w;
  const uint16_t* W; int64_t groups, kc, w_bstride;
  float* out; int64_t ld_o, o_bstride;
  int32_t* dev_info;
  char* ws;
};
size_t softmax_product_ws(int64_t n, int64_t V, int64_t cols);
hipError_t launch_softmax_product(const SoftmaxProductArgs& a);
// the same product in one pass over the logits (online softmax), one pass per 64 columns
size_t softmax_product_online_ws(int64_t n, int64_t V, int64_t cols);
hipError_t launch_softmax_product_online(const SoftmaxProductArgs& a);

struct CreditArgs {
  hipStream_t stream;
  int64_t nb, n, d, k;
  const float* e; int64_t ld_e;
  const float* vk; int64_t v_bstride;
  const float* credit_b; int64_t b_bstride;
  const float* a_w;
  float* y_out; int64_t y_bstride;
  loca_mb* mb_out;
  char* ws;
};
size_t credit_from_top_error_ws(int64_t nb, int64_t n, int64_t k);
hipError_t launch_credit_from_top_error(const CreditArgs& a);

struct StatsArgs {
  hipStream_t stream;
  int64_t nb, n, d, k;
  const void* x; loca_dtype x_dtype; int64_t ldx, x_bstride;
  const float* y; int64_t y_bstride; const float* a_w;
  double eta; loca_mb* mb;
  void* S; void* K; loca_dtype acc; int64_t s_bstride, k_bstride;
  int32_t* dev_info;
  char* ws;
  bool overwrite;  // S and K are written, not accumulated into
};
size_t accumulate_stats_ws(int64_t nb, int64_t n, int64_t d, int64_t k, loca_dtype acc);
hipError_t launch_accumulate_stats(const StatsArgs& a);

struct SolveArgs {
  hipStream_t stream;
  int64_t nb, d, k;
  const void* S; const void* K; loca_dtype acc; int64_t s_bstride, k_bstride;
  const float* lp; const float* rp; int64_t r_prev, lp_bstride, rp_bstride;
  const double* lambdas; int64_t n_lambda;
  float* m_out; int64_t m_bstride;
  const float* credit_b; int64_t b_bstride;
  float* w_dense_out; int64_t w_bstride;
  int32_t* dev_info; char* ws;
  // Internal (acc = F64 only): the factor and the scaling of a previous call with the same
  // S, lambdas, sizes and workspace, ordered before this one, are still in `ws`; only the
  // right-hand sides are scaled, carried through the forward substitution and solved.
  // dev_info then reads 0: the factor's status is the one the factoring call reported.
  bool reuse_factor;
};
size_t ridge_solve_ws(int64_t nb, int64_t d, int64_t m, int64_t n_lambda, loca_dtype acc);
hipError_t launch_ridge_solve(const SolveArgs& a);

struct TruncArgs {
  hipStream_t stream;
  int64_t nm, d, kp, r_a;
  const float* m; int64_t m_bstride;
  const float* r; int64_t r_bstride, r_group;
  float* a_out; int64_t a_bstride;
  float* b_out; int64_t b_bstride;
  float* sigma_out; int64_t sigma_bstride;
  float* w_dense_out; int64_t w_bstride;
  int32_t* dev_info; char* ws;
};
size_t lowrank_truncate_ws(int64_t nm, int64_t d, int64_t kp, int64_t r_a);
hipError_t launch_lowrank_truncate(const TruncArgs& a);

struct ProjArgs {
  hipStream_t stream;
  int64_t nb, d, k, r_a;
  const void* S; const void* K; loca_dtype acc; int64_t s_bstride, k_bstride;
  const float* credit_b; int64_t b_bstride;
  const float* proj_a; int64_t pa_bstride;
  const float* b_cur; int64_t bc_bstride;
  const double* lambdas; int64_t n_lambda;
  float* b_out; int64_t bo_bstride; float* g_out;
  int32_t* dev_info; char* ws;
};
size_t projected_ws(int64_t nb, int64_t d, int64_t k, int64_t r_a, int64_t n_lambda);
hipError_t launch_ridge_solve_projected(const ProjArgs& a);

struct CalibArgs {
  hipStream_t stream;
  int64_t nb, d, np_, k;
  const float* e; const float* g; int64_t g_bstride;
  double beta;
  const void* wu; loca_dtype wu_dtype; int64_t vocab;
  float* bt_out; int64_t bt_bstride;
  float* at_out; int64_t at_bstride;
  float* vk_out; int64_t vk_bstride;
  float* sigma_out; double* alpha_out;
  int32_t* dev_info; char* ws;
  bool primal;  // primal form (a Cholesky solve in d unknowns) instead of the dual one
  // subspace-iteration form (loca_feedback_fit_large): basis width, power iterations and
  // the caller's start block (d x l float)
  int64_t l, q;
  const float* omega;
};
size_t feedback_fit_ws(int64_t nb, int64_t d, int64_t np_, int64_t k);
size_t feedback_fit_primal_ws(int64_t nb, int64_t d, int64_t np_, int64_t k);
size_t feedback_fit_large_ws(int64_t nb, int64_t d, int64_t np_, int64_t k, int64_t l);
hipError_t launch_feedback_fit_large(const CalibArgs& a);
// The rank-k truncation of F_b = M_b R_b and the Stage I credit factors (shared by the fits);
// returns U_k^T (k x d) and V_k S_k (d x k) per block, both inside the workspace.
size_t calib_factor_ws(int64_t nb, int64_t d, int64_t kp, int64_t k);
hipError_t launch_calib_factors(const CalibArgs& a, const float* M, int64_t m_bs, const float* R, int64_t r_bs,
                                int64_t r_group, int64_t kp, char* ws, float** ut, float** vs);

// Realisation error of the fitted adapters (Section S6).
struct FitArgs {
  hipStream_t stream;
  int64_t nb, d, k, r_prev;
  const float* m; int64_t m_bstride;
  const float* r; int64_t r_bstride;
  const void* K; loca_dtype acc; int64_t k_bstride;
  const float* lp; int64_t lp_bstride;
  const loca_mb* mb_log; int64_t n_mb;
  const double* lambdas; int64_t n_lambda;
  double* out;
  char* ws;
};
size_t realization_error_ws(int64_t nb, int64_t d, int64_t k, int64_t r_prev, int64_t n_lambda);
hipError_t launch_realization_error(const FitArgs& a);
hipError_t launch_feedback_fit(const CalibArgs& a);

hipError_t launch_dense_targets(hipStream_t s, int64_t nb, int64_t n, int64_t k, int64_t d,
                                const float* y, int64_t y_bstride, const loca_mb* mb,
                                const float* credit_b, int64_t b_bstride, float* t_out,
                                int64_t t_bstride);
// out (rows x cols) = L (rows x kk, ld kk) * R (kk x cols, ld cols), float, batched.
hipError_t launch_lowrank_product(hipStream_t s, int64_t nmat, int64_t rows, int64_t cols,
                                  int64_t kk, const float* L, int64_t l_bstride, int64_t l_ld,
                                  const float* R, int64_t r_bstride, int64_t r_group, int64_t r_ld,
                                  float* out, int64_t out_bstride);

// The fused LM head ("Local Targets", Eq. 4; Section S11): out = E Vm with the logits formed
// in-kernel and never stored.
constexpr int kMaxFusedSplits = 64;  // vocabulary ranges combined per token
struct FusedArgs {
  hipStream_t stream;
  int64_t n, V, d, c;
  const uint16_t* h; int64_t ldh;
  const uint16_t* wu;
  const int32_t* labels; const float* w;
  const uint16_t* vm; int64_t ld_vm;
  float* out; int64_t ld_out;
  int32_t* dev_info; char* ws;
};
size_t fused_head_ws(int64_t n, int64_t V, int64_t c);
hipError_t launch_fused_head(const FusedArgs& a);

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }
}  // namespace loca
