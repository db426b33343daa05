// k_subspace.hip -- Stage I calibration for probe counts beyond the hidden width
// (Section S5: the feedback ridge fit of Eq. 5, the theorem on its solution and the
// rank-truncation lemma).
//
// With Np > d probes the fitted map F_hat_b = G_b E^T (E E^T + beta I)^{-1} is a full-rank
// d x d matrix, so its best rank-k approximation is not available from a small factored
// product.  It is taken here by randomised subspace iteration on the factored map
// F_hat_b = G_b R, R = E^T (E E^T + beta I)^{-1} (Np x d), which never forms F_hat_b:
//   1. S_E = E E^T (d x d, float64 products of the float probes);
//   2. R^T = (S_E + beta I)^{-1} E by the library's float64 Cholesky solve, in chunks of at
//      most 128 right-hand sides (the primal form of the theorem; shared by the blocks);
//   3. from the caller's start block Omega (d x l), q rounds of
//        Y = orth(F_hat Omega),  Omega = orth(F_hat^T Y),
//      then Q = orth(F_hat Omega) and B^T = F_hat^T Q; every product with F_hat or F_hat^T
//      is two skinny products (R^T Omega, then G_b times it; G_b^T Y, then R^T-side), float64;
//      orth is Cholesky QR taken twice (the Gram in float64, its factor inverted in one
//      workgroup, the basis multiplied by L^{-T});
//   4. the rank-k truncation of the Ritz approximation Q B (kp = l) with the factored
//      truncation of the hot path, then the credit factors as for the small-probe fits;
//   5. the alignment diagnostic alpha_b = <U_k^T G_b, S_k V_k^T E> / (||S_k V_k^T E|| ||G_b||).
// The leading k Ritz pairs converge to those of F_hat at the rate (sigma_{l+1} / sigma_k)^(2q+1)
// of subspace iteration with l columns.
#include "loca_launch.h"

namespace loca {

namespace {

constexpr int kT = 256;
constexpr int kMaxL = 128;
constexpr int kSolveCols = 128;  // right-hand sides per Cholesky solve

// C_z (m x n, row-major, ldc) = sum_p A_z(i, p) B_z(p, j) in float64, p in increasing order;
// A_z(i, p) = A[z a_bs + i a_si + p a_sp], B_z(p, j) = B[z b_bs + p b_sp + j b_sj].
// 64 x 64 tiles of C, 16-deep chunks of p through LDS; each thread holds 4 x 4 outputs at
// rows ty + 16 r and columns tx + 16 c.  The staging walks the operand's unit-stride index
// fastest.  Grid: (n tiles, m tiles, batch).
template <typename AT, typename BT>
__global__ __launch_bounds__(kT) void k_gemm64(int64_t m, int64_t n, int64_t K, const AT* __restrict__ A,
                                               int64_t a_bs, int64_t a_si, int64_t a_sp, const BT* __restrict__ B,
                                               int64_t b_bs, int64_t b_sp, int64_t b_sj, double* __restrict__ C,
                                               int64_t c_bs, int64_t ldc) {
  __shared__ double sA[16][65];
  __shared__ double sB[16][65];
  const int64_t z = blockIdx.z;
  const int64_t i0 = (int64_t)blockIdx.y * 64, j0 = (int64_t)blockIdx.x * 64;
  const AT* Az = A + z * a_bs;
  const BT* Bz = B + z * b_bs;
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
  const bool a_pf = a_sp == 1;
  const bool b_pf = b_sp == 1 && b_sj != 1;
  double acc[4][4];
#pragma unroll
  for (int r = 0; r < 4; ++r)
#pragma unroll
    for (int c = 0; c < 4; ++c) acc[r][c] = 0.0;
  for (int64_t p0 = 0; p0 < K; p0 += 16) {
    for (int e = tid; e < 1024; e += kT) {
      const int pa = a_pf ? (e & 15) : (e >> 6), ia = a_pf ? (e >> 4) : (e & 63);
      const int64_t gi = i0 + ia, gpa = p0 + pa;
      sA[pa][ia] = (gi < m && gpa < K) ? (double)Az[gi * a_si + gpa * a_sp] : 0.0;
      const int pb = b_pf ? (e & 15) : (e >> 6), jb = b_pf ? (e >> 4) : (e & 63);
      const int64_t gj = j0 + jb, gpb = p0 + pb;
      sB[pb][jb] = (gj < n && gpb < K) ? (double)Bz[gpb * b_sp + gj * b_sj] : 0.0;
    }
    __syncthreads();
#pragma unroll
    for (int p = 0; p < 16; ++p) {
      double av[4], bv[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) av[r] = sA[p][ty + 16 * r];
#pragma unroll
      for (int c = 0; c < 4; ++c) bv[c] = sB[p][tx + 16 * c];
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[r][c] = fma(av[r], bv[c], acc[r][c]);
    }
    __syncthreads();
  }
  double* Cz = C + z * c_bs;
#pragma unroll
  for (int r = 0; r < 4; ++r)
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int64_t gi = i0 + ty + 16 * r, gj = j0 + tx + 16 * c;
      if (gi < m && gj < n) Cz[gi * ldc + gj] = acc[r][c];
    }
}

// Per batch entry z: G_z (l x l, float64, symmetric, row-major) + shift_rel tr(G_z) I = L L^T,
// and U_z = L^{-T} (upper triangular).  One workgroup; the factor lives in LDS.  A pivot that
// is not positive (the basis lost rank, or non-finite data) is replaced by 1, and
// flag[z] becomes LOCA_INFO_BASIS_RANK unless it already holds a code.
__global__ __launch_bounds__(kT) void k_chol_inv(int l, const double* __restrict__ G, double shift_rel,
                                                 double* __restrict__ U, int32_t* __restrict__ flag) {
  __shared__ double sA[kMaxL][kMaxL + 1];
  __shared__ double sD[kMaxL];
  __shared__ double red[kT / 64];
  __shared__ double sh;
  __shared__ int bad;
  const int tid = threadIdx.x;
  const int64_t z = blockIdx.x;
  const double* Gz = G + z * l * l;
  double tr = 0.0;
  for (int i = tid; i < l; i += kT) tr += Gz[(int64_t)i * l + i];
  tr = block_sum(tr, red);
  if (tid == 0) {
    sh = shift_rel * tr;
    bad = 0;
  }
  __syncthreads();
  for (int e = tid; e < l * l; e += kT) {
    const int i = e / l, j = e % l;
    sA[i][j] = Gz[e] + (i == j ? sh : 0.0);
  }
  __syncthreads();
  // right-looking Cholesky on the lower triangle
  for (int j = 0; j < l; ++j) {
    if (tid == 0) {
      double piv = sA[j][j];
      if (!(piv > 0.0)) {
        bad = 1;
        piv = 1.0;
      }
      sA[j][j] = sqrt(piv);
    }
    __syncthreads();
    for (int i = j + 1 + tid; i < l; i += kT) sA[i][j] /= sA[j][j];
    __syncthreads();
    const int rem = l - j - 1;
    for (int e = tid; e < rem * rem; e += kT) {
      const int i = j + 1 + e / rem, c = j + 1 + e % rem;
      if (c <= i) sA[i][c] -= sA[i][j] * sA[c][j];
    }
    __syncthreads();
  }
  // column jj of L^{-1} by forward substitution, kept in row jj above the diagonal (entries
  // the factor does not use) and its diagonal in sD: each thread writes only its own row
  for (int jj = tid; jj < l; jj += kT) {
    const double xd = 1.0 / sA[jj][jj];
    sD[jj] = xd;
    for (int i = jj + 1; i < l; ++i) {
      double s = sA[i][jj] * xd;
      for (int p = jj + 1; p < i; ++p) s += sA[i][p] * sA[jj][p];
      sA[jj][i] = -s / sA[i][i];
    }
  }
  __syncthreads();
  double* Uz = U + z * l * l;
  for (int e = tid; e < l * l; e += kT) {
    const int p = e / l, i = e % l;  // U(p, i) = (L^{-1})(i, p)
    Uz[e] = i > p ? sA[p][i] : (i == p ? sD[p] : 0.0);
  }
  if (tid == 0 && bad) atomicCAS(&flag[z], 0, LOCA_INFO_BASIS_RANK);
}

// dst (d x w, float64) = columns c0 .. c0 + w - 1 of E (d x np, float)
__global__ void k_cols_f64(int64_t d, int64_t np_, int64_t c0, int w, int wh, const float* __restrict__ E,
                           double* __restrict__ dst) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= d * w) return;
  const int64_t c = e / w, j = e % w;
  dst[e] = j < wh ? (double)E[c * np_ + c0 + j] : 0.0;
}
// columns c0 .. c0 + wh - 1 of Rt (d x np) = the first wh columns of M (d x w)
__global__ void k_cols_put(int64_t d, int64_t np_, int64_t c0, int w, int wh, const float* __restrict__ M,
                           float* __restrict__ Rt) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= d * wh) return;
  const int64_t c = e / wh, j = e % wh;
  Rt[c * np_ + c0 + j] = M[c * w + j];
}
// per block b: dst_b (d x l, float64) = Omega (d x l, float)
__global__ void k_start_block(int64_t cnt, const float* __restrict__ omega, double* __restrict__ dst) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e < cnt) dst[(int64_t)blockIdx.y * cnt + e] = (double)omega[e];
}
// out = (float) in, element by element
__global__ void k_f64_f32(int64_t cnt, const double* __restrict__ in, float* __restrict__ out) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e < cnt) out[e] = (float)in[e];
}
// per block: out_b (l x d, float) = in_b^T (in_b: d x l, float64)
__global__ void k_f64_f32_t(int64_t d, int l, const double* __restrict__ in, float* __restrict__ out) {
  const int64_t b = blockIdx.y;
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= d * l) return;
  const int64_t j = e / d, c = e % d;
  out[b * d * l + e] = (float)in[b * d * l + c * l + j];
}
// dev_info[b] = the first non-zero status of the nch solves (the solves serve every block)
__global__ void k_fold_solve_info(const int32_t* __restrict__ sinfo, int nch, int32_t* __restrict__ dev_info,
                                  int64_t nb) {
  int32_t v = 0;
  for (int h = 0; h < nch && v == 0; ++h) v = sinfo[h];
  for (int64_t b = threadIdx.x; b < nb; b += blockDim.x) dev_info[b] = v;
}
// alpha_b = <P_b, Q_b> / (||Q_b|| ||G_b||), P_b and Q_b k x np (float64), G_b d x np (float).
// One workgroup per block: strided per-thread sums in a fixed order, then a fixed tree.
__global__ __launch_bounds__(kT) void k_alpha_dense(int64_t kn, int64_t dn, const double* __restrict__ P,
                                                    const double* __restrict__ Q, const float* __restrict__ G,
                                                    int64_t g_bs, double* __restrict__ alpha_out) {
  __shared__ double red[3][kT / 64];
  const int64_t b = blockIdx.x;
  double pq = 0.0, qq = 0.0, gg = 0.0;
  for (int64_t e = threadIdx.x; e < kn; e += kT) {
    const double p = P[b * kn + e], q = Q[b * kn + e];
    pq += p * q;
    qq += q * q;
  }
  for (int64_t e = threadIdx.x; e < dn; e += kT) {
    const double g = (double)G[b * g_bs + e];
    gg += g * g;
  }
  pq = block_sum(pq, red[0]);
  qq = block_sum(qq, red[1]);
  gg = block_sum(gg, red[2]);
  if (threadIdx.x == 0) {
    const double den = sqrt(qq) * sqrt(gg);
    alpha_out[b] = den > 0.0 ? pq / den : 0.0;
  }
}

inline unsigned cdiv(int64_t a, int64_t b) { return (unsigned)((a + b - 1) / b); }

template <typename AT, typename BT>
void gemm(hipStream_t st, int64_t nbat, int64_t m, int64_t n, int64_t K, const AT* A, int64_t a_bs, int64_t a_si,
          int64_t a_sp, const BT* B, int64_t b_bs, int64_t b_sp, int64_t b_sj, double* C, int64_t c_bs, int64_t ldc) {
  k_gemm64<AT, BT><<<dim3(cdiv(n, 64), cdiv(m, 64), (unsigned)nbat), kT, 0, st>>>(m, n, K, A, a_bs, a_si, a_sp, B,
                                                                                 b_bs, b_sp, b_sj, C, c_bs, ldc);
}

}  // namespace

size_t feedback_fit_large_ws(int64_t nb, int64_t d, int64_t np_, int64_t k, int64_t l) {
  const int64_t w = np_ < kSolveCols ? np_ : kSolveCols, nch = (np_ + kSolveCols - 1) / kSolveCols;
  size_t s = align256(sizeof(double) * d * d);         // S_E
  s += align256(sizeof(double) * d * w);               // a chunk of E (float64 right-hand sides)
  s += align256(sizeof(float) * d * w);                // its solution
  s += align256(sizeof(int32_t) * nch);                // the solves' status
  s += ridge_solve_ws(1, d, w, 1, LOCA_F64);
  s += align256(sizeof(float) * d * np_);              // R^T
  s += 2 * align256(sizeof(double) * nb * d * l);      // the two d x l blocks per block
  s += align256(sizeof(double) * nb * np_ * l);        // the np x l products
  s += 2 * align256(sizeof(double) * nb * l * l);      // Gram and L^{-T}
  s += align256(sizeof(float) * nb * d * l);           // Q (float)
  s += align256(sizeof(float) * nb * l * d);           // B = Q^T F_hat (float)
  s += 2 * align256(sizeof(double) * nb * k * np_);    // U_k^T G and S_k V_k^T E
  return s + calib_factor_ws(nb, d, l, k);
}

hipError_t launch_feedback_fit_large(const CalibArgs& a) {
  const int64_t d = a.d, np_ = a.np_, k = a.k, nb = a.nb, l = a.l;
  const int64_t w = np_ < kSolveCols ? np_ : kSolveCols, nch = (np_ + kSolveCols - 1) / kSolveCols;
  hipStream_t st = a.stream;
  char* p = a.ws;
  double* SE = (double*)p; p += align256(sizeof(double) * d * d);
  double* Ec = (double*)p; p += align256(sizeof(double) * d * w);
  float* Mc = (float*)p; p += align256(sizeof(float) * d * w);
  int32_t* sinfo = (int32_t*)p; p += align256(sizeof(int32_t) * nch);
  char* sws = p; p += ridge_solve_ws(1, d, w, 1, LOCA_F64);
  float* Rt = (float*)p; p += align256(sizeof(float) * d * np_);
  double* X0 = (double*)p; p += align256(sizeof(double) * nb * d * l);
  double* X1 = (double*)p; p += align256(sizeof(double) * nb * d * l);
  double* T = (double*)p; p += align256(sizeof(double) * nb * np_ * l);
  double* Gm = (double*)p; p += align256(sizeof(double) * nb * l * l);
  double* U = (double*)p; p += align256(sizeof(double) * nb * l * l);
  float* Qf = (float*)p; p += align256(sizeof(float) * nb * d * l);
  float* Bf = (float*)p; p += align256(sizeof(float) * nb * l * d);
  double* Pa = (double*)p; p += align256(sizeof(double) * nb * k * np_);
  double* Qa = (double*)p; p += align256(sizeof(double) * nb * k * np_);
  hipError_t e;

  // 1-2: S_E = E E^T, then R^T = (S_E + beta I)^{-1} E chunk by chunk: the first chunk
  // factors S_E + beta I, the later ones reuse that factor (same width w, the last chunk's
  // missing columns zero; their status entries read 0, the factor's is the first)
  gemm<float, float>(st, 1, d, d, np_, a.e, 0, np_, 1, a.e, 0, 1, np_, SE, 0, d);
  const double lam[1] = {a.beta};
  for (int64_t h = 0; h < nch; ++h) {
    const int64_t c0 = h * kSolveCols;
    const int wh = (int)(np_ - c0 < kSolveCols ? np_ - c0 : kSolveCols);
    k_cols_f64<<<cdiv(d * w, 256), 256, 0, st>>>(d, np_, c0, (int)w, wh, a.e, Ec);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    SolveArgs sa{st, 1, d, w, SE, Ec, LOCA_F64, d * d, d * w, nullptr, nullptr, 0, 0, 0, lam, 1, Mc, d * w,
                 nullptr, 0, nullptr, 0, sinfo + h, sws, h > 0};
    if ((e = launch_ridge_solve(sa)) != hipSuccess) return e;
    k_cols_put<<<cdiv(d * wh, 256), 256, 0, st>>>(d, np_, c0, (int)w, wh, Mc, Rt);
  }
  k_fold_solve_info<<<1, 64, 0, st>>>(sinfo, (int)nch, a.dev_info, nb);
  if ((e = hipGetLastError()) != hipSuccess) return e;

  // products with the factored map, per block (batch z = block):
  // dst = F_hat src = G (R src), with R src = (R^T)^T src (np x l)
  auto fwd = [&](const double* src, double* dst) {
    gemm<float, double>(st, nb, np_, l, d, Rt, 0, 1, np_, src, d * l, l, 1, T, np_ * l, l);
    gemm<float, double>(st, nb, d, l, np_, a.g, a.g_bstride, np_, 1, T, np_ * l, l, 1, dst, d * l, l);
  };
  // dst = F_hat^T src = R^T (G^T src)
  auto bwd = [&](const double* src, double* dst) {
    gemm<float, double>(st, nb, np_, l, d, a.g, a.g_bstride, 1, np_, src, d * l, l, 1, T, np_ * l, l);
    gemm<float, double>(st, nb, d, l, np_, Rt, 0, np_, 1, T, np_ * l, l, 1, dst, d * l, l);
  };
  // X = orth(X) by two passes of Cholesky QR (tmp is overwritten; the result ends in X)
  auto orth = [&](double* X, double* tmp) {
    double* src = X;
    double* dst = tmp;
    for (int pass = 0; pass < 2; ++pass) {
      gemm<double, double>(st, nb, l, l, d, src, d * l, 1, l, src, d * l, l, 1, Gm, l * l, l);
      k_chol_inv<<<(unsigned)nb, kT, 0, st>>>((int)l, Gm, pass == 0 ? 1e-14 : 0.0, U, a.dev_info);
      gemm<double, double>(st, nb, d, l, l, src, d * l, l, 1, U, l * l, l, 1, dst, d * l, l);
      double* t = src;
      src = dst;
      dst = t;
    }
  };

  // 3: subspace iteration from the caller's start block
  k_start_block<<<dim3(cdiv(d * l, 256), (unsigned)nb), 256, 0, st>>>(d * l, a.omega, X0);
  for (int64_t it = 0; it < a.q; ++it) {
    fwd(X0, X1);
    orth(X1, X0);
    bwd(X1, X0);
    orth(X0, X1);
  }
  fwd(X0, X1);
  orth(X1, X0);  // Q in X1
  bwd(X1, X0);   // B^T = F_hat^T Q in X0
  if ((e = hipGetLastError()) != hipSuccess) return e;

  // 4: truncation of Q B (per block: M = Q, R = B) and the credit factors
  k_f64_f32<<<cdiv(nb * d * l, 256), 256, 0, st>>>(nb * d * l, X1, Qf);
  k_f64_f32_t<<<dim3(cdiv(d * l, 256), (unsigned)nb), 256, 0, st>>>(d, (int)l, X0, Bf);
  float *ut = nullptr, *vs = nullptr;
  if ((e = launch_calib_factors(a, Qf, d * l, Bf, l * d, 1, l, p, &ut, &vs)) != hipSuccess) return e;

  // 5: P = U_k^T G (k x np) and Q = (V_k S_k)^T E (k x np), then alpha
  gemm<float, float>(st, nb, k, np_, d, ut, k * d, d, 1, a.g, a.g_bstride, np_, 1, Pa, k * np_, np_);
  gemm<float, float>(st, nb, k, np_, d, vs, d * k, 1, k, a.e, 0, np_, 1, Qa, k * np_, np_);
  k_alpha_dense<<<(unsigned)nb, kT, 0, st>>>(k * np_, d * np_, Pa, Qa, a.g, a.g_bstride, a.alpha_out);
  return hipGetLastError();
}

}  // namespace loca
