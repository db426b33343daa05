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

// C_z (m x n, row-major, ldc) = sum_p A_z(i, p) B_z(p, j) in float64;
// A_z(i, p) = A[z a_bs + i a_si + p a_sp], B_z(p, j) = B[z b_bs + p b_sp + j b_sj].
// 64 x 64 tiles of C, 16-deep chunks of p through LDS (two buffers; the next chunk is loaded
// into registers while the current one is used); each thread holds 4 x 4 outputs at rows
// ty + 16 r and columns tx + 16 c.  The staging walks the operand's unit-stride index
// fastest.  With nsplit > 1 the p range is cut into nsplit equal ranges of whole chunks
// (p in increasing order inside each), and range s writes its sum to
// part + ((z nsplit + s) m + i) n + j instead of C; k_sum_parts then adds the ranges in
// order.  Grid: (n tiles, m tiles, batch x nsplit).
template <typename AT, typename BT>
__global__ __launch_bounds__(kT) __attribute__((amdgpu_waves_per_eu(4))) void k_gemm64(
    int64_t m, int64_t n, int64_t K, const AT* __restrict__ A,
                                               int64_t a_bs, int64_t a_si, int64_t a_sp, const BT* __restrict__ B,
                                               int64_t b_bs, int64_t b_sp, int64_t b_sj, double* __restrict__ C,
                                               int64_t c_bs, int64_t ldc, int nsplit, int64_t kchunk,
                                               double* __restrict__ part) {
  __shared__ double sA[2][16][65];
  __shared__ double sB[2][16][65];
  const int64_t z = blockIdx.z / nsplit, sp = blockIdx.z % nsplit;
  const int64_t i0 = (int64_t)blockIdx.y * 64, j0 = (int64_t)blockIdx.x * 64;
  const int64_t kb = sp * kchunk, ke = kb + kchunk < K ? kb + kchunk : K;
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
  // per staged element u: its LDS slot and its operand's address at p = 0 (rows and columns
  // past the matrix read as zeros)
  const AT* pa_[4];
  const BT* pb_[4];
  int la[4], lb[4], qa[4], qb[4];
  bool oka[4], okb[4];
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int e = tid + u * kT;
    const int pa = a_pf ? (e & 15) : (e >> 6), ia = a_pf ? (e >> 4) : (e & 63);
    const int pb = b_pf ? (e & 15) : (e >> 6), jb = b_pf ? (e >> 4) : (e & 63);
    oka[u] = i0 + ia < m;
    okb[u] = j0 + jb < n;
    pa_[u] = Az + (oka[u] ? (i0 + ia) * a_si : 0) + pa * a_sp;
    pb_[u] = Bz + (okb[u] ? (j0 + jb) * b_sj : 0) + pb * b_sp;
    qa[u] = pa;
    qb[u] = pb;
    la[u] = pa * 65 + ia;
    lb[u] = pb * 65 + jb;
  }
  double ra[4], rb[4];
  auto load = [&](int64_t p0) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      ra[u] = (oka[u] && p0 + qa[u] < ke) ? (double)pa_[u][p0 * a_sp] : 0.0;
      rb[u] = (okb[u] && p0 + qb[u] < ke) ? (double)pb_[u][p0 * b_sp] : 0.0;
    }
  };
  auto store = [&](int buf) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      (&sA[buf][0][0])[la[u]] = ra[u];
      (&sB[buf][0][0])[lb[u]] = rb[u];
    }
  };
  if (kb < ke) {
    load(kb);
    store(0);
  }
  __syncthreads();
  int cur = 0;
  for (int64_t p0 = kb; p0 < ke; p0 += 16) {
    const bool more = p0 + 16 < ke;
    if (more) load(p0 + 16);
#pragma unroll 4
    for (int p = 0; p < 16; ++p) {
      double av[4], bv[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) av[r] = sA[cur][p][ty + 16 * r];
#pragma unroll
      for (int c = 0; c < 4; ++c) bv[c] = sB[cur][p][tx + 16 * c];
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[r][c] = fma(av[r], bv[c], acc[r][c]);
    }
    if (more) store(cur ^ 1);
    __syncthreads();
    cur ^= 1;
  }
  double* Cz = nsplit > 1 ? part + (z * nsplit + sp) * m * n : C + z * c_bs;
  const int64_t ld = nsplit > 1 ? n : ldc;
#pragma unroll
  for (int r = 0; r < 4; ++r)
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int64_t gi = i0 + ty + 16 * r, gj = j0 + tx + 16 * c;
      if (gi < m && gj < n) Cz[gi * ld + gj] = acc[r][c];
    }
}

// C_z[i][j] = sum over s = 0 .. nsplit - 1 in order of part_(z, s)[i][j]
__global__ void k_sum_parts(int64_t m, int64_t n, int nsplit, const double* __restrict__ part,
                            double* __restrict__ C, int64_t c_bs, int64_t ldc) {
  const int64_t z = blockIdx.y;
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= m * n) return;
  const double* pz = part + z * nsplit * m * n + e;
  double v = 0.0;
  for (int s = 0; s < nsplit; ++s) v += pz[(int64_t)s * m * n];
  C[z * c_bs + (e / n) * ldc + e % n] = v;
}

// Per batch entry z: G_z (l x l, float64, symmetric, row-major) + shift_rel tr(G_z) I = U^T U
// (U upper triangular, U = L^T of the lower Cholesky factor) and U_z = U^{-1} (upper
// triangular), so that X U^{-1} has the Gram identity.  One workgroup per entry; the matrix
// lives in registers: thread (ty, tx) of a 16 x 16 grid owns the entries
// (ty + 16 i, tx + 16 c).  Step j of the factorization needs only row j of the partly
// reduced matrix, which its owners publish to a double-buffered LDS row (one barrier per
// step); the inverse is then built bottom-up the same way (row i of U^{-1} is final once the
// rows below it have been applied), with U in LDS for its column reads.  A pivot that is not
// positive (the basis lost rank, or non-finite data) is replaced by 1, and flag[z] becomes
// LOCA_INFO_BASIS_RANK unless it already holds a code.
__global__ __launch_bounds__(kT) void k_chol_inv(int l, const double* __restrict__ G, double shift_rel,
                                                 double* __restrict__ U, int32_t* __restrict__ flag) {
  constexpr int NI = kMaxL / 16;
  __shared__ double rowbuf[2][kMaxL];
  __shared__ double sU[kMaxL][kMaxL + 1];
  __shared__ double red[kT / 64];
  const int tid = threadIdx.x, ty = tid >> 4, tx = tid & 15;
  const int64_t z = blockIdx.x;
  const double* Gz = G + z * l * l;
  double tr = 0.0;
  for (int i = tid; i < l; i += kT) tr += Gz[(int64_t)i * l + i];
  tr = block_sum(tr, red);
  const double sh = shift_rel * tr;
  double a[NI][NI];
#pragma unroll
  for (int i = 0; i < NI; ++i)
#pragma unroll
    for (int c = 0; c < NI; ++c) {
      const int r = ty + 16 * i, q = tx + 16 * c;
      a[i][c] = (r < l && q < l && q >= r) ? Gz[(int64_t)r * l + q] + (q == r ? sh : 0.0) : 0.0;
    }
  if (ty == 0)
#pragma unroll
    for (int c = 0; c < NI; ++c) rowbuf[0][tx + 16 * c] = a[0][c];
  bool bad = false;
  for (int j = 0; j < l; ++j) {
    __syncthreads();
    const double* rb = rowbuf[j & 1];
    double piv = rb[j];
    if (!(piv > 0.0)) {
      bad = true;
      piv = 1.0;
    }
    const double ujj = sqrt(piv);
    const double inv = 1.0 / ujj;
    double ur[NI], uc[NI];
#pragma unroll
    for (int i = 0; i < NI; ++i) ur[i] = rb[(ty + 16 * i) & (kMaxL - 1)] * inv;
#pragma unroll
    for (int c = 0; c < NI; ++c) uc[c] = rb[(tx + 16 * c) & (kMaxL - 1)] * inv;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int r = ty + 16 * i;
      if (r == j) {  // owners of row j: the final row of U
#pragma unroll
        for (int c = 0; c < NI; ++c) {
          const int q = tx + 16 * c;
          if (q >= j && q < l) a[i][c] = (q == j) ? ujj : uc[c];
        }
      } else if (r > j && r < l) {
#pragma unroll
        for (int c = 0; c < NI; ++c) {
          const int q = tx + 16 * c;
          if (q >= r && q < l) a[i][c] -= ur[i] * uc[c];
        }
      }
    }
    if (j + 1 < l) {
#pragma unroll
      for (int i = 0; i < NI; ++i)
        if (ty + 16 * i == j + 1)
#pragma unroll
          for (int c = 0; c < NI; ++c) rowbuf[(j + 1) & 1][tx + 16 * c] = a[i][c];
    }
  }
#pragma unroll
  for (int i = 0; i < NI; ++i)
#pragma unroll
    for (int c = 0; c < NI; ++c) sU[ty + 16 * i][tx + 16 * c] = a[i][c];
  __syncthreads();
  // X = U^{-1} bottom-up: t holds the partial sums sum_{k > i0} U[r][k] X[k][c] of rows r < i0
  double t[NI][NI];
#pragma unroll
  for (int i = 0; i < NI; ++i)
#pragma unroll
    for (int c = 0; c < NI; ++c) t[i][c] = 0.0;
  {
    const int last = l - 1;
#pragma unroll
    for (int i = 0; i < NI; ++i)
      if (ty + 16 * i == last)
#pragma unroll
        for (int c = 0; c < NI; ++c) {
          const int q = tx + 16 * c;
          const double x = (q == last) ? 1.0 / sU[last][last] : 0.0;
          t[i][c] = x;
          rowbuf[last & 1][q] = x;
        }
  }
  for (int i0 = l - 1; i0 >= 0; --i0) {
    __syncthreads();
    const double* xb = rowbuf[i0 & 1];
    double xc[NI];
#pragma unroll
    for (int c = 0; c < NI; ++c) xc[c] = xb[tx + 16 * c];
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int r = ty + 16 * i;
      if (r < i0) {
        const double uri = sU[r][i0];
#pragma unroll
        for (int c = 0; c < NI; ++c) t[i][c] += uri * xc[c];
      }
    }
    const int nr = i0 - 1;  // the row finished in this step
    if (nr >= 0) {
      const double rinv = 1.0 / sU[nr][nr];
#pragma unroll
      for (int i = 0; i < NI; ++i)
        if (ty + 16 * i == nr)
#pragma unroll
          for (int c = 0; c < NI; ++c) {
            const int q = tx + 16 * c;
            const double x = (q >= nr && q < l) ? ((q == nr ? 1.0 : 0.0) - t[i][c]) * rinv : 0.0;
            t[i][c] = x;
            rowbuf[nr & 1][q] = x;
          }
    }
  }
  double* Uz = U + z * l * l;
#pragma unroll
  for (int i = 0; i < NI; ++i)
#pragma unroll
    for (int c = 0; c < NI; ++c) {
      const int r = ty + 16 * i, q = tx + 16 * c;
      if (r < l && q < l) Uz[(int64_t)r * l + q] = (q >= r) ? t[i][c] : 0.0;
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
// out = (double) in, element by element
__global__ void k_f32_f64(int64_t cnt, const float* __restrict__ in, double* __restrict__ out) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e < cnt) out[e] = (double)in[e];
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
// alpha_b = <P_b, Q_b> / (||Q_b|| ||G_b||), P_b and Q_b k x np (float64), G_b d x np (float),
// in two passes: workgroup (s, b) sums slice s of kAlphaParts equal slices of P_b Q_b, Q_b Q_b
// and G_b G_b (strided per-thread sums, then a fixed tree), and one workgroup per block adds
// the slices in order.
constexpr int kAlphaParts = 256;
__global__ __launch_bounds__(kT) void k_alpha_part(int64_t kn, int64_t dn, const double* __restrict__ P,
                                                   const double* __restrict__ Q, const float* __restrict__ G,
                                                   int64_t g_bs, double* __restrict__ part) {
  __shared__ double red[3][kT / 64];
  const int64_t b = blockIdx.y, s = blockIdx.x;
  const int64_t ks = (kn + kAlphaParts - 1) / kAlphaParts, ds = (dn + kAlphaParts - 1) / kAlphaParts;
  const int64_t k0 = s * ks, k1 = k0 + ks < kn ? k0 + ks : kn;
  const int64_t d0 = s * ds, d1 = d0 + ds < dn ? d0 + ds : dn;
  double pq = 0.0, qq = 0.0, gg = 0.0;
  for (int64_t e = k0 + threadIdx.x; e < k1; e += kT) {
    const double p = P[b * kn + e], q = Q[b * kn + e];
    pq += p * q;
    qq += q * q;
  }
  for (int64_t e = d0 + threadIdx.x; e < d1; e += kT) {
    const double g = (double)G[b * g_bs + e];
    gg += g * g;
  }
  pq = block_sum(pq, red[0]);
  qq = block_sum(qq, red[1]);
  gg = block_sum(gg, red[2]);
  if (threadIdx.x == 0) {
    double* o = part + (b * kAlphaParts + s) * 3;
    o[0] = pq;
    o[1] = qq;
    o[2] = gg;
  }
}
__global__ __launch_bounds__(64) void k_alpha_sum(const double* __restrict__ part, double* __restrict__ alpha_out) {
  const int64_t b = blockIdx.x;
  if (threadIdx.x != 0) return;
  double pq = 0.0, qq = 0.0, gg = 0.0;
  for (int s = 0; s < kAlphaParts; ++s) {
    const double* o = part + (b * kAlphaParts + s) * 3;
    pq += o[0];
    qq += o[1];
    gg += o[2];
  }
  const double den = sqrt(qq) * sqrt(gg);
  alpha_out[b] = den > 0.0 ? pq / den : 0.0;
}

inline unsigned cdiv(int64_t a, int64_t b) { return (unsigned)((a + b - 1) / b); }

// The p range is split when the output tiles alone would leave most of the chip idle:
// about kGemmWaves workgroups in all, ranges of at least 64, partial sums within kPartElems.
constexpr int64_t kGemmWaves = 768;
constexpr int64_t kPartElems = (int64_t)4 << 20;
template <typename AT, typename BT>
void gemm(hipStream_t st, double* part, int64_t nbat, int64_t m, int64_t n, int64_t K, const AT* A, int64_t a_bs,
          int64_t a_si, int64_t a_sp, const BT* B, int64_t b_bs, int64_t b_sp, int64_t b_sj, double* C, int64_t c_bs,
          int64_t ldc) {
  const int64_t tiles = (int64_t)cdiv(n, 64) * cdiv(m, 64) * nbat;
  int64_t ns = (kGemmWaves + tiles - 1) / tiles;
  if (ns > K / 64) ns = K / 64;
  if (ns > kPartElems / (nbat * m * n)) ns = kPartElems / (nbat * m * n);
  if (ns < 1) ns = 1;
  const int64_t kc = ((K + ns - 1) / ns + 15) / 16 * 16;
  ns = (K + kc - 1) / kc;
  k_gemm64<AT, BT><<<dim3(cdiv(n, 64), cdiv(m, 64), (unsigned)(nbat * ns)), kT, 0, st>>>(
      m, n, K, A, a_bs, a_si, a_sp, B, b_bs, b_sp, b_sj, C, c_bs, ldc, (int)ns, kc, part);
  if (ns > 1)
    k_sum_parts<<<dim3(cdiv(m * n, 256), (unsigned)nbat), 256, 0, st>>>(m, n, (int)ns, part, C, c_bs, ldc);
}

}  // namespace

size_t feedback_fit_large_ws(int64_t nb, int64_t d, int64_t np_, int64_t k, int64_t l) {
  const int64_t w = np_ < kSolveCols ? np_ : kSolveCols, nch = (np_ + kSolveCols - 1) / kSolveCols;
  const int64_t wm = w > l ? w : l;
  size_t s = align256(sizeof(double) * d * d);         // S_E
  s += align256(sizeof(double) * d * w);               // a chunk of E (float64 right-hand sides)
  s += align256(sizeof(float) * d * wm);               // a solution
  s += align256(sizeof(int32_t) * (nch > 2 ? nch : 2));  // the solves' status
  s += ridge_solve_ws(1, d, wm, 1, LOCA_F64);
  s += align256(sizeof(float) * d * np_);              // R^T
  s += 2 * align256(sizeof(double) * nb * d * l);      // the two d x l blocks per block
  s += align256(sizeof(double) * nb * np_ * l);        // the np x l products
  s += 2 * align256(sizeof(double) * nb * l * l);      // Gram and L^{-T}
  s += align256(sizeof(float) * nb * d * l);           // Q (float)
  s += align256(sizeof(float) * nb * l * d);           // B = Q^T F_hat (float)
  s += 2 * align256(sizeof(double) * nb * k * np_);    // U_k^T G and S_k V_k^T E
  s += align256(sizeof(double) * nb * kAlphaParts * 3);  // the alignment's partial sums
  s += align256(sizeof(double) * kPartElems);           // partial sums of split products
  return s + calib_factor_ws(nb, d, l, k);
}

hipError_t launch_feedback_fit_large(const CalibArgs& a) {
  const int64_t d = a.d, np_ = a.np_, k = a.k, nb = a.nb, l = a.l;
  const int64_t w = np_ < kSolveCols ? np_ : kSolveCols, nch = (np_ + kSolveCols - 1) / kSolveCols;
  const int64_t wm = w > l ? w : l;
  hipStream_t st = a.stream;
  char* p = a.ws;
  double* SE = (double*)p; p += align256(sizeof(double) * d * d);
  double* Ec = (double*)p; p += align256(sizeof(double) * d * w);
  float* Mc = (float*)p; p += align256(sizeof(float) * d * wm);
  int32_t* sinfo = (int32_t*)p; p += align256(sizeof(int32_t) * (nch > 2 ? nch : 2));
  char* sws = p; p += ridge_solve_ws(1, d, wm, 1, LOCA_F64);
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
  double* Ap = (double*)p; p += align256(sizeof(double) * nb * kAlphaParts * 3);
  double* Pt = (double*)p; p += align256(sizeof(double) * kPartElems);
  hipError_t e;

  // 1-2: S_E = E E^T; S_E + beta I is factored once by the first solve below and every
  // later solve reuses that factor (same width, the status of a reusing solve reads 0).
  // R enters the products in one of two ways, whichever takes fewer solves:
  //   formed: R^T = (S_E + beta I)^{-1} E in chunks of w columns (the last chunk's missing
  //           columns zero), shared by the blocks: ceil(np / w) solves;
  //   applied: R src = E^T ((S_E + beta I)^{-1} src) and R^T src' = (S_E + beta I)^{-1} (E src')
  //           with a solve of l columns per block and product: 2 (q + 1) nb solves.
  gemm<float, float>(st, Pt, 1, d, d, np_, a.e, 0, np_, 1, a.e, 0, 1, np_, SE, 0, d);
  const double lam[1] = {a.beta};
  const bool applied = 2 * (a.q + 1) * nb < nch;
  int nsolve = 0;
  // Mc (d x l, float) = (S_E + beta I)^{-1} K (d x l, float64); the factoring solve's status
  // goes to every block's dev_info before anything else can write there
  auto solve_l = [&](const double* K) {
    SolveArgs sa{st, 1, d, l, SE, K, LOCA_F64, d * d, d * l, nullptr, nullptr, 0, 0, 0, lam, 1, Mc, d * l,
                 nullptr, 0, nullptr, 0, sinfo + (nsolve > 0 ? 1 : 0), sws, nsolve > 0};
    hipError_t r = launch_ridge_solve(sa);
    if (r == hipSuccess && nsolve == 0) {
      k_fold_solve_info<<<1, 64, 0, st>>>(sinfo, 1, a.dev_info, nb);
      r = hipGetLastError();
    }
    ++nsolve;
    return r;
  };
  for (int64_t h = 0; h < (applied ? 0 : nch); ++h) {
    const int64_t c0 = h * kSolveCols;
    const int wh = (int)(np_ - c0 < kSolveCols ? np_ - c0 : kSolveCols);
    k_cols_f64<<<cdiv(d * w, 256), 256, 0, st>>>(d, np_, c0, (int)w, wh, a.e, Ec);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    SolveArgs sa{st, 1, d, w, SE, Ec, LOCA_F64, d * d, d * w, nullptr, nullptr, 0, 0, 0, lam, 1, Mc, d * w,
                 nullptr, 0, nullptr, 0, sinfo + h, sws, h > 0};
    if ((e = launch_ridge_solve(sa)) != hipSuccess) return e;
    k_cols_put<<<cdiv(d * wh, 256), 256, 0, st>>>(d, np_, c0, (int)w, wh, Mc, Rt);
  }
  if (!applied) {
    k_fold_solve_info<<<1, 64, 0, st>>>(sinfo, (int)nch, a.dev_info, nb);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }

  // products with the factored map, per block (batch z = block); a failed solve launch
  // is kept in se and ends the call after the iteration
  hipError_t se = hipSuccess;
  // dst = F_hat src = G (R src), R src (np x l) into T
  auto fwd = [&](const double* src, double* dst) {
    if (!applied) {
      gemm<float, double>(st, Pt, nb, np_, l, d, Rt, 0, 1, np_, src, d * l, l, 1, T, np_ * l, l);
    } else {
      for (int64_t b = 0; b < nb && se == hipSuccess; ++b) {
        if ((se = solve_l(src + b * d * l)) != hipSuccess) break;
        gemm<float, float>(st, Pt, 1, np_, l, d, a.e, 0, 1, np_, Mc, 0, l, 1, T + b * np_ * l, 0, l);
      }
    }
    gemm<float, double>(st, Pt, nb, d, l, np_, a.g, a.g_bstride, np_, 1, T, np_ * l, l, 1, dst, d * l, l);
  };
  // dst = F_hat^T src = R^T (G^T src), G^T src (np x l) into T
  auto bwd = [&](const double* src, double* dst) {
    gemm<float, double>(st, Pt, nb, np_, l, d, a.g, a.g_bstride, 1, np_, src, d * l, l, 1, T, np_ * l, l);
    if (!applied) {
      gemm<float, double>(st, Pt, nb, d, l, np_, Rt, 0, np_, 1, T, np_ * l, l, 1, dst, d * l, l);
    } else {
      // dst = E T first (the solve's right-hand side), then its solution over it
      gemm<float, double>(st, Pt, nb, d, l, np_, a.e, 0, np_, 1, T, np_ * l, l, 1, dst, d * l, l);
      for (int64_t b = 0; b < nb && se == hipSuccess; ++b) {
        if ((se = solve_l(dst + b * d * l)) != hipSuccess) break;
        k_f32_f64<<<cdiv(d * l, 256), 256, 0, st>>>(d * l, Mc, dst + b * d * l);
      }
    }
  };
  // X = orth(X) by two passes of Cholesky QR (tmp is overwritten; the result ends in X)
  auto orth = [&](double* X, double* tmp) {
    double* src = X;
    double* dst = tmp;
    for (int pass = 0; pass < 2; ++pass) {
      gemm<double, double>(st, Pt, nb, l, l, d, src, d * l, 1, l, src, d * l, l, 1, Gm, l * l, l);
      k_chol_inv<<<(unsigned)nb, kT, 0, st>>>((int)l, Gm, pass == 0 ? 1e-14 : 0.0, U, a.dev_info);
      gemm<double, double>(st, Pt, nb, d, l, l, src, d * l, l, 1, U, l * l, l, 1, dst, d * l, l);
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
  if (se != hipSuccess) return se;
  if ((e = hipGetLastError()) != hipSuccess) return e;

  // 4: truncation of Q B (per block: M = Q, R = B) and the credit factors
  k_f64_f32<<<cdiv(nb * d * l, 256), 256, 0, st>>>(nb * d * l, X1, Qf);
  k_f64_f32_t<<<dim3(cdiv(d * l, 256), (unsigned)nb), 256, 0, st>>>(d, (int)l, X0, Bf);
  float *ut = nullptr, *vs = nullptr;
  if ((e = launch_calib_factors(a, Qf, d * l, Bf, l * d, 1, l, p, &ut, &vs)) != hipSuccess) return e;

  // 5: P = U_k^T G (k x np) and Q = (V_k S_k)^T E (k x np), then alpha
  gemm<float, float>(st, Pt, nb, k, np_, d, ut, k * d, d, 1, a.g, a.g_bstride, np_, 1, Pa, k * np_, np_);
  gemm<float, float>(st, Pt, nb, k, np_, d, vs, d * k, 1, k, a.e, 0, np_, 1, Qa, k * np_, np_);
  k_alpha_part<<<dim3((unsigned)kAlphaParts, (unsigned)nb), kT, 0, st>>>(k * np_, d * np_, Pa, Qa, a.g,
                                                                         a.g_bstride, Ap);
  k_alpha_sum<<<(unsigned)nb, 64, 0, st>>>(Ap, a.alpha_out);
  return hipGetLastError();
}

}  // namespace loca
