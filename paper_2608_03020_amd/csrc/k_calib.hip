// k_calib.hip -- one-time Stage I calibration of the feedback map (Section S5).
//
// The feedback ridge fit of Eq. 5, F_hat = argmin ||F E - G||_F^2 + beta ||F||_F^2 for the
// probe columns E (top errors, d x Np, shared by the blocks) and G_b (exact gradients at
// block b, d x Np), in its dual form (Section S5's theorem): F_hat = G_b (E^T E + beta I)^{-1} E^T,
// evaluated as a Cholesky solve in Np unknowns:
//   1. Gamma = E^T E (fp64, split over the rows of E, fixed-order sums);
//   2. Gamma + beta I = L L^T (one workgroup, fp64);
//   3. R = (Gamma + beta I)^{-1} E^T (Np x d), one column of E^T per thread (forward and
//      back substitution with L);
//   4. the best rank-k approximation F_b = U_k S_k V_k^T of F_hat = G_b R (the rank-
//      truncation lemma of Section S5) with the factored Eckart-Young truncation of the
//      hot path (M = G_b, right factor R shared by all blocks);
//   5. the credit factors B~ = S_k U_k^T, A~ = W_u V_k (W_u^T folded into A~, as on the hot
//      path), and the alignment diagnostic alpha_b = <F_b E, G_b> / (||F_b E|| ||G_b||),
//      with ||F_b E|| = ||S_k V_k^T E|| since U_k has orthonormal columns.
//
// The realisation error of a fitted adapter (Section S6) is also here: it needs the same
// fixed-order products of tall d x (<= 64) operands.
#include "loca_launch.h"

namespace loca {

namespace {

constexpr int kT = 256;
constexpr int kMaxNp = 64;
constexpr int kRows = 32;

// part[(b * ns + z) * kL * kR + j * kR + n] = sum_{c in rows of z} L_b(c, j) R_b(c, n), fp64,
// L_b(c, j) = L[b * l_bs + c * l_sc + j * l_sj] (likewise R); rows split in ns equal ranges
// of 32-row multiples (grid: x = z, y = b).
template <typename RT>
__global__ __launch_bounds__(kT) void k_tall_cross(int64_t d, int kL, int kR, const float* __restrict__ L,
                                                   int64_t l_bs, int64_t l_sc, int64_t l_sj,
                                                   const RT* __restrict__ R, int64_t r_bs, int64_t r_sc,
                                                   int64_t r_sn, int ns, double* __restrict__ part) {
  __shared__ double sL[kRows][kMaxNp + 1];
  __shared__ double sR[kRows][kMaxNp + 1];
  const int64_t b = blockIdx.y;
  const int z = blockIdx.x;
  const int64_t chunk = ((d + ns - 1) / ns + kRows - 1) / kRows * kRows;
  const int64_t ib = (int64_t)z * chunk, ie = ib + chunk < d ? ib + chunk : d;
  const float* Lb = L + b * l_bs;
  const RT* Rb = R + b * r_bs;
  const int nout = kL * kR;
  double acc[(kMaxNp * kMaxNp) / kT];
#pragma unroll
  for (int q = 0; q < (kMaxNp * kMaxNp) / kT; ++q) acc[q] = 0.0;
  for (int64_t i0 = ib; i0 < ie; i0 += kRows) {
    __syncthreads();
    for (int e = threadIdx.x; e < kRows * kMaxNp; e += kT) {
      const int r = e / kMaxNp, c = e % kMaxNp;
      const int64_t i = i0 + r;
      sL[r][c] = (i < ie && c < kL) ? (double)Lb[i * l_sc + c * l_sj] : 0.0;
      sR[r][c] = (i < ie && c < kR) ? (double)Rb[i * r_sc + c * r_sn] : 0.0;
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < (kMaxNp * kMaxNp) / kT; ++q) {
      const int e = threadIdx.x + kT * q;
      if (e < nout) {
        const int j = e / kR, n = e % kR;
        double s = acc[q];
        for (int r = 0; r < kRows; ++r) s += sL[r][j] * sR[r][n];
        acc[q] = s;
      }
    }
  }
  double* out = part + (b * ns + z) * (int64_t)nout;
#pragma unroll
  for (int q = 0; q < (kMaxNp * kMaxNp) / kT; ++q) {
    const int e = threadIdx.x + kT * q;
    if (e < nout) out[e] = acc[q];
  }
}

// Lmat = chol(sum_z part_z + beta I) (lower, np x np, fp64, row-major), one workgroup.
__global__ __launch_bounds__(kT) void k_chol_small(int np_, int ns, const double* __restrict__ part, double beta,
                                                   double* __restrict__ Lmat, int32_t* __restrict__ dev_info,
                                                   int64_t nb) {
  __shared__ double sA[kMaxNp][kMaxNp + 1];
  const int tid = threadIdx.x;
  for (int e = tid; e < np_ * np_; e += kT) {
    const int i = e / np_, j = e % np_;
    double s = 0.0;
    for (int z = 0; z < ns; ++z) s += part[(int64_t)z * np_ * np_ + e];
    sA[i][j] = s + (i == j ? beta : 0.0);
  }
  __syncthreads();
  for (int j = 0; j < np_; ++j) {
    if (tid == 0) {
      const double piv = sA[j][j];
      if (!(piv > 0.0))
        for (int64_t b = 0; b < nb; ++b) atomicCAS(&dev_info[b], 0, j + 1);
      sA[j][j] = sqrt(piv);
    }
    __syncthreads();
    for (int i = j + 1 + tid; i < np_; i += kT) sA[i][j] /= sA[j][j];
    __syncthreads();
    for (int e = tid; e < (np_ - j - 1) * (np_ - j - 1); e += kT) {
      const int i = j + 1 + e / (np_ - j - 1), c = j + 1 + e % (np_ - j - 1);
      if (c <= i) sA[i][c] -= sA[i][j] * sA[c][j];
    }
    __syncthreads();
  }
  for (int e = tid; e < np_ * np_; e += kT) {
    const int i = e / np_, j = e % np_;
    Lmat[e] = j <= i ? sA[i][j] : 0.0;
  }
}

// R[:, c] = (L L^T)^{-1} E[c, :]^T for every column c < d (thread per column; R is np x d).
__global__ __launch_bounds__(kT) void k_ridge_cols(int64_t d, int np_, const float* __restrict__ E,
                                                   const double* __restrict__ Lmat, float* __restrict__ R) {
  __shared__ double sL[kMaxNp * kMaxNp];
  for (int e = threadIdx.x; e < np_ * np_; e += kT) sL[e] = Lmat[e];
  __syncthreads();
  const int64_t c = (int64_t)blockIdx.x * kT + threadIdx.x;
  if (c >= d) return;
  double y[kMaxNp];
#pragma unroll
  for (int i = 0; i < kMaxNp; ++i) y[i] = i < np_ ? (double)E[c * np_ + i] : 0.0;
  // forward: L y' = e
#pragma unroll
  for (int i = 0; i < kMaxNp; ++i) {
    if (i < np_) {
      double s = y[i];
#pragma unroll
      for (int j = 0; j < i; ++j) s -= sL[i * np_ + j] * y[j];
      y[i] = s / sL[i * np_ + i];
    }
  }
  // back: L^T x = y'
#pragma unroll
  for (int i = kMaxNp - 1; i >= 0; --i) {
    if (i < np_) {
      double s = y[i];
#pragma unroll
      for (int j = i + 1; j < kMaxNp; ++j)
        if (j < np_) s -= sL[j * np_ + i] * y[j];
      y[i] = s / sL[i * np_ + i];
    }
  }
#pragma unroll
  for (int i = 0; i < kMaxNp; ++i)
    if (i < np_) R[(int64_t)i * d + c] = (float)y[i];
}

// Per block: B~ = S_k U_k^T from U_k^T (a) and sigma; V_k = (V_k S_k) / S_k from b (zero where
// sigma = 0), kept for A~.  Grid: x over d, y = block.
__global__ void k_calib_factors(int64_t d, int k, int np_, const float* __restrict__ a, const float* __restrict__ bvs,
                                const float* __restrict__ sigma, float* __restrict__ bt_out, int64_t bt_bstride,
                                float* __restrict__ vk) {
  const int64_t b = blockIdx.y;
  const int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= d) return;
  for (int j = 0; j < k; ++j) {
    const float s = sigma[b * np_ + j];
    bt_out[b * bt_bstride + (int64_t)j * d + c] = s * a[(b * k + j) * d + c];
    vk[(b * d + c) * k + j] = s > 0.f ? bvs[(b * d + c) * k + j] / s : 0.f;
  }
}

// alpha_b = <P, Q> / (||Q|| ||G||) from the fixed-order sums of the partial products
// P = U_k^T G, Q = S_k V_k^T E (k x np) and ||G||^2, taken over the probe columns in chunks of
// at most 64 (chunk h: columns 64 h .. 64 h + w_h - 1, partials of P and Q at
// pP + h * nb * ns * k * 64 with row length w_h, those of G_h^T G_h at pG2 + h * nb * ns * 64 * 64).
// One workgroup per block: thread e sums entry e over the row ranges in order, then
// fixed-order workgroup sums.
__global__ __launch_bounds__(kT) void k_calib_alpha(int64_t nb, int k, int np_, int ns, const double* __restrict__ pP,
                                                    const double* __restrict__ pQ, const double* __restrict__ pG2,
                                                    double* __restrict__ alpha_out) {
  __shared__ double red[3][kT / 64];
  const int64_t b = blockIdx.x;
  double pq = 0.0, qq = 0.0, gg = 0.0;
  for (int h = 0; h * kMaxNp < np_; ++h) {
    const int w = np_ - h * kMaxNp < kMaxNp ? np_ - h * kMaxNp : kMaxNp;
    const double* P = pP + (int64_t)h * nb * ns * k * kMaxNp;
    const double* Q = pQ + (int64_t)h * nb * ns * k * kMaxNp;
    const double* G2 = pG2 + (int64_t)h * nb * ns * kMaxNp * kMaxNp;
    for (int e = threadIdx.x; e < k * w; e += kT) {
      double p = 0.0, q = 0.0;
      for (int z = 0; z < ns; ++z) {
        p += P[(b * ns + z) * k * w + e];
        q += Q[(b * ns + z) * k * w + e];
      }
      pq += p * q;
      qq += q * q;
    }
    for (int e = threadIdx.x; e < w; e += kT)
      for (int z = 0; z < ns; ++z) gg += G2[(b * ns + z) * w * w + e * w + e];
  }
  pq = block_sum(pq, red[0]);
  qq = block_sum(qq, red[1]);
  gg = block_sum(gg, red[2]);
  if (threadIdx.x == 0) {
    const double den = sqrt(qq) * sqrt(gg);
    alpha_out[b] = den > 0.0 ? pq / den : 0.0;
  }
}

// Primal form helpers.  S_E = E E^T (d x d, fp64, both triangles) from the rows of E
// (d x np, row-major): one thread per entry on or above the diagonal, products of floats
// summed in fp64 in the order of the probes, the mirror written too.
__global__ void k_rows_gram(int64_t d, int np_, const float* __restrict__ E, double* __restrict__ S) {
  const int64_t i = blockIdx.y;
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (j < i || j >= d) return;
  const float* ei = E + i * np_;
  const float* ej = E + j * np_;
  double s = 0.0;
  for (int p = 0; p < np_; ++p) s += (double)ei[p] * (double)ej[p];
  S[i * d + j] = s;
  S[j * d + i] = s;
}
// out (fp64) = in (float), element by element
__global__ void k_to_f64(int64_t cnt, const float* __restrict__ in, double* __restrict__ out) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e < cnt) out[e] = (double)in[e];
}
// R (np x d) = Rt^T (Rt: d x np), 32 x 32 tiles through LDS
__global__ void k_transpose_f32(int64_t d, int np_, const float* __restrict__ Rt, float* __restrict__ R) {
  __shared__ float t[32][33];
  const int64_t c0 = (int64_t)blockIdx.x * 32, p0 = (int64_t)blockIdx.y * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;  // 256 threads: 32 x 8
  for (int r = ty; r < 32; r += 8) {
    const int64_t c = c0 + r, p = p0 + tx;
    t[r][tx] = (c < d && p < np_) ? Rt[c * np_ + p] : 0.f;
  }
  __syncthreads();
  for (int r = ty; r < 32; r += 8) {
    const int64_t p = p0 + r, c = c0 + tx;
    if (p < np_ && c < d) R[p * d + c] = t[tx][r];
  }
}

// A~_b = W_u V_k,b (vocab x k, k <= 64) on the fp32 matrix cores (v_mfma_f32_32x32x2f32):
// a workgroup of four waves takes 128 rows of W_u, wave w rows 32 w .. 32 w + 31 and all k
// columns in two 32-wide blocks; d is walked in slices of 64 staged through LDS (W_u as
// floats, exact for bf16 input), the next slice loaded into registers while the current one
// is multiplied.  Grid: x over 128-row tiles, y = block.
constexpr int kFoldR = 128, kFoldK = 64;
template <typename WT>
__global__ __launch_bounds__(kT) void k_head_fold(int64_t vocab, int64_t d, int k, const WT* __restrict__ wu,
                                                  const float* __restrict__ vk, float* __restrict__ at_out,
                                                  int64_t at_bstride) {
  __shared__ float sW[kFoldR][kFoldK + 1];
  __shared__ float sB[kFoldK][kFoldK + 1];
  const int64_t b = blockIdx.y;
  const int64_t v0 = (int64_t)blockIdx.x * kFoldR;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const float* Vb = vk + b * d * k;
  constexpr int NW = kFoldR * kFoldK / kT, NB = kFoldK * kFoldK / kT;  // elements per thread
  float rw[NW], rb[NB];
  auto gload = [&](int64_t k0) {
#pragma unroll
    for (int t = 0; t < NW; ++t) {
      const int e = tid + kT * t, r = e / kFoldK, c = e % kFoldK;
      rw[t] = (v0 + r < vocab && k0 + c < d) ? load_as_f32(wu + (v0 + r) * d + k0 + c) : 0.f;
    }
#pragma unroll
    for (int t = 0; t < NB; ++t) {
      const int e = tid + kT * t, r = e / kFoldK, c = e % kFoldK;
      rb[t] = (k0 + r < d && c < k) ? Vb[(k0 + r) * k + c] : 0.f;
    }
  };
  f32x16_t acc[2];
#pragma unroll
  for (int q = 0; q < 2; ++q)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[q][r] = 0.f;
  const int nq = k > 32 ? 2 : 1;
  gload(0);
  for (int64_t k0 = 0; k0 < d; k0 += kFoldK) {
    __syncthreads();  // the previous slice's readers are done
#pragma unroll
    for (int t = 0; t < NW; ++t) {
      const int e = tid + kT * t;
      sW[e / kFoldK][e % kFoldK] = rw[t];
    }
#pragma unroll
    for (int t = 0; t < NB; ++t) {
      const int e = tid + kT * t;
      sB[e / kFoldK][e % kFoldK] = rb[t];
    }
    __syncthreads();
    if (k0 + kFoldK < d) gload(k0 + kFoldK);
    // A lane l = W[row l % 32][kk + l / 32], B lane l = V_k[kk + l / 32][col l % 32]
#pragma unroll 8
    for (int kk = 0; kk < kFoldK; kk += 2) {
      const float a = sW[32 * wid + (lane & 31)][kk + (lane >> 5)];
      acc[0] = mfma_f32x2(a, sB[kk + (lane >> 5)][lane & 31], acc[0]);
      if (nq > 1) acc[1] = mfma_f32x2(a, sB[kk + (lane >> 5)][32 + (lane & 31)], acc[1]);
    }
  }
#pragma unroll
  for (int q = 0; q < 2; ++q)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int64_t row = v0 + 32 * wid + mfma32_row(lane, r);
      const int col = 32 * q + (lane & 31);
      if (row < vocab && col < k) at_out[b * at_bstride + row * k + col] = acc[q][r];
    }
}

// vk_out[b][c][j] = V_k (the internal copy, d x k per block, packed)
__global__ void k_copy_vk(int64_t d, int k, const float* __restrict__ vk, float* __restrict__ out, int64_t bstride) {
  const int64_t b = blockIdx.y;
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e < d * k) out[b * bstride + e] = vk[b * d * k + e];
}

// the primal form's single solve serves every block: its status goes to each block's dev_info
__global__ void k_copy_info(const int32_t* __restrict__ src, int32_t* __restrict__ dst, int64_t nb) {
  for (int64_t b = threadIdx.x; b < nb; b += blockDim.x) dst[b] = src[0];
}

__global__ void k_zero_i32(int32_t* p, int64_t cnt) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < cnt) p[i] = 0;
}

int calib_splits(int64_t d) {
  const int64_t s = d / 256;
  return (int)(s < 1 ? 1 : (s > 16 ? 16 : s));
}

// ------------------------------------------------------------------ realisation error
// Per (block b, lambda l), from fixed-order sums of the tall products' partials (z ranges):
//   tZ = tr((M^T K)(B~ R^T)) - tr((Lp^T K)(B~ Rp^T)),   tW = tr((M^T M)(R R^T)) - tr((Lp^T M)(R Rp^T)),
//   t2 = sum_m eta_bar_m^2 ||Q_m||^2,   out = {t2 - tZ - lam tW, t2, tr((M^T M)(R R^T))}.
// B~ R^T and R Rp^T are rows / columns of R R^T, since R = [Rp; B~].
template <typename F>
LOCA_DEV double zsum_block(F term, int cnt, double* sred) {
  double v = 0.0;
  for (int e = threadIdx.x; e < cnt; e += kT) v += term(e);
  return block_sum(v, sred);  // thread 0
}
__global__ __launch_bounds__(kT) void k_fit_finalize(int64_t nb, int nl, int kp, int k, int rp, int ns,
                                                     const double* __restrict__ pMK, const double* __restrict__ pMM,
                                                     const double* __restrict__ pRR, const double* __restrict__ pLK,
                                                     const double* __restrict__ pLM, const loca_mb* __restrict__ mb_log,
                                                     int64_t n_mb, const double* __restrict__ lam,
                                                     double* __restrict__ out) {
  __shared__ double sred[kT / 64];
  const int64_t mi = blockIdx.x;
  const int64_t b = mi / nl;
  const int l = (int)(mi % nl);
  // partial z of entry e of a product with `cnt` entries, for launch-local block index bl
  auto zs = [&](const double* part, int64_t bl, int64_t cnt, int e) {
    double v = 0.0;
    for (int z = 0; z < ns; ++z) v += part[(bl * ns + z) * cnt + e];
    return v;
  };
  const double* MK = pMK + (int64_t)l * nb * ns * kp * k;
  const double* MM = pMM + (int64_t)l * nb * ns * kp * kp;
  const double* LM = pLM + (int64_t)l * nb * ns * rp * kp;
  const double z1 = zsum_block([&](int e) {
    const int a = e / k, c = e % k;
    return zs(MK, b, (int64_t)kp * k, e) * zs(pRR, b, (int64_t)kp * kp, (rp + c) * kp + a);
  }, kp * k, sred);
  __syncthreads();
  const double w1 = zsum_block([&](int e) {
    const int a = e / kp, a2 = e % kp;
    return zs(MM, b, (int64_t)kp * kp, e) * zs(pRR, b, (int64_t)kp * kp, a2 * kp + a);
  }, kp * kp, sred);
  __syncthreads();
  double z2 = 0.0, w2 = 0.0;
  if (rp > 0) {
    z2 = zsum_block([&](int e) {
      const int q = e / k, c = e % k;
      return zs(pLK, b, (int64_t)rp * k, e) * zs(pRR, b, (int64_t)kp * kp, (rp + c) * kp + q);
    }, rp * k, sred);
    __syncthreads();
    w2 = zsum_block([&](int e) {
      const int q = e / kp, a = e % kp;
      return zs(LM, b, (int64_t)rp * kp, e) * zs(pRR, b, (int64_t)kp * kp, a * kp + q);
    }, rp * kp, sred);
  }
  if (threadIdx.x == 0) {
    double t2 = 0.0;
    for (int64_t m = 0; m < n_mb; ++m) {
      const loca_mb& r = mb_log[m * nb + b];
      t2 += r.eta_bar * r.eta_bar * r.sum_q2;
    }
    out[3 * mi + 0] = t2 - (z1 - z2) - lam[l] * (w1 - w2);
    out[3 * mi + 1] = t2;
    out[3 * mi + 2] = w1;
  }
}

struct FitLams {
  double v[8];
};
__global__ void k_fit_lams(FitLams l, double* out, int cnt) {
  if ((int)threadIdx.x < cnt) out[threadIdx.x] = l.v[threadIdx.x];
}

}  // namespace

size_t realization_error_ws(int64_t nb, int64_t d, int64_t k, int64_t r_prev, int64_t n_lambda) {
  const int64_t ns = calib_splits(d), kp = r_prev + k;
  size_t s = 256;  // lambdas
  s += align256(sizeof(double) * n_lambda * nb * ns * kp * k);       // M^T K
  s += align256(sizeof(double) * n_lambda * nb * ns * kp * kp);      // M^T M
  s += align256(sizeof(double) * nb * ns * kp * kp);                 // R R^T
  s += align256(sizeof(double) * nb * ns * (r_prev > 0 ? r_prev : 1) * k);               // Lp^T K
  s += align256(sizeof(double) * n_lambda * nb * ns * (r_prev > 0 ? r_prev : 1) * kp);   // Lp^T M
  return s;
}

hipError_t launch_realization_error(const FitArgs& a) {
  const int64_t d = a.d, k = a.k, rp = a.r_prev, kp = rp + k, nb = a.nb, nl = a.n_lambda;
  const int ns = calib_splits(d);
  char* p = a.ws;
  double* dlam = (double*)p; p += 256;
  double* pMK = (double*)p; p += align256(sizeof(double) * nl * nb * ns * kp * k);
  double* pMM = (double*)p; p += align256(sizeof(double) * nl * nb * ns * kp * kp);
  double* pRR = (double*)p; p += align256(sizeof(double) * nb * ns * kp * kp);
  double* pLK = (double*)p; p += align256(sizeof(double) * nb * ns * (rp > 0 ? rp : 1) * k);
  double* pLM = (double*)p;
  hipStream_t st = a.stream;
  FitLams fl;
  for (int i = 0; i < 8; ++i) fl.v[i] = i < nl ? a.lambdas[i] : 0.0;
  k_fit_lams<<<1, 64, 0, st>>>(fl, dlam, (int)nl);
  const dim3 g((unsigned)ns, (unsigned)nb);
  // R R^T from the rows of R (R^T(c, j) = R[j][c])
  k_tall_cross<float><<<g, kT, 0, st>>>(d, (int)kp, (int)kp, a.r, a.r_bstride, 1, d, a.r, a.r_bstride, 1, d, ns, pRR);
  if (rp > 0) {
    if (a.acc == LOCA_F64)
      k_tall_cross<double><<<g, kT, 0, st>>>(d, (int)rp, (int)k, a.lp, a.lp_bstride, rp, 1, (const double*)a.K,
                                             a.k_bstride, k, 1, ns, pLK);
    else
      k_tall_cross<float><<<g, kT, 0, st>>>(d, (int)rp, (int)k, a.lp, a.lp_bstride, rp, 1, (const float*)a.K,
                                            a.k_bstride, k, 1, ns, pLK);
  }
  for (int64_t l = 0; l < nl; ++l) {
    const float* Ml = a.m + l * a.m_bstride;  // matrix (b, l) at m + (b nl + l) m_bstride
    const int64_t mbs = nl * a.m_bstride;
    double* oMK = pMK + l * nb * ns * kp * k;
    double* oMM = pMM + l * nb * ns * kp * kp;
    if (a.acc == LOCA_F64)
      k_tall_cross<double><<<g, kT, 0, st>>>(d, (int)kp, (int)k, Ml, mbs, kp, 1, (const double*)a.K, a.k_bstride, k,
                                             1, ns, oMK);
    else
      k_tall_cross<float><<<g, kT, 0, st>>>(d, (int)kp, (int)k, Ml, mbs, kp, 1, (const float*)a.K, a.k_bstride, k,
                                            1, ns, oMK);
    k_tall_cross<float><<<g, kT, 0, st>>>(d, (int)kp, (int)kp, Ml, mbs, kp, 1, Ml, mbs, kp, 1, ns, oMM);
    if (rp > 0)
      k_tall_cross<float><<<g, kT, 0, st>>>(d, (int)rp, (int)kp, a.lp, a.lp_bstride, rp, 1, Ml, mbs, kp, 1, ns,
                                            pLM + l * nb * ns * rp * kp);
  }
  k_fit_finalize<<<(unsigned)(nb * nl), kT, 0, st>>>(nb, (int)nl, (int)kp, (int)k, (int)rp, ns, pMK, pMM, pRR, pLK,
                                                     pLM, a.mb_log, a.n_mb, dlam, a.out);
  return hipGetLastError();
}

// The rank-k truncation of F_b = M_b R_b (kp columns; R_b shared by r_group consecutive
// blocks) and the credit factors of Stage I: B~, V_k and the folded head A~.  Workspace:
// U_k^T (k x d), V_k S_k and V_k (d x k) per block, the truncation's status and its own.
size_t calib_factor_ws(int64_t nb, int64_t d, int64_t kp, int64_t k) {
  size_t s = align256(sizeof(float) * nb * k * d);                // U_k^T
  s += align256(sizeof(float) * nb * d * k);                      // V_k S_k
  s += align256(sizeof(float) * nb * d * k);                      // V_k
  s += align256(sizeof(int32_t) * nb);                             // the truncation's own status
  s += lowrank_truncate_ws(nb, d, kp, k);
  return s;
}

hipError_t launch_calib_factors(const CalibArgs& a, const float* M, int64_t m_bs, const float* R, int64_t r_bs,
                                int64_t r_group, int64_t kp, char* p, float** ut_out, float** vs_out) {
  const int64_t d = a.d, k = a.k, nb = a.nb;
  float* ut = (float*)p; p += align256(sizeof(float) * nb * k * d);
  float* vs = (float*)p; p += align256(sizeof(float) * nb * d * k);
  float* vk = (float*)p; p += align256(sizeof(float) * nb * d * k);
  int32_t* tinfo = (int32_t*)p; p += align256(sizeof(int32_t) * nb);
  hipStream_t st = a.stream;
  // the truncation's status array is private: its only writes are zeros
  TruncArgs t{st, nb, d, kp, k, M, m_bs, R, r_bs, r_group, ut, k * d, vs, d * k, a.sigma_out, kp, nullptr, 0,
              tinfo, p};
  hipError_t e = launch_lowrank_truncate(t);
  if (e != hipSuccess) return e;
  k_calib_factors<<<dim3((unsigned)((d + 255) / 256), (unsigned)nb), 256, 0, st>>>(
      d, (int)k, (int)kp, ut, vs, a.sigma_out, a.bt_out, a.bt_bstride, vk);
  if (a.vk_out) {
    dim3 g((unsigned)((d * k + 255) / 256), (unsigned)nb);
    k_copy_vk<<<g, 256, 0, st>>>(d, (int)k, vk, a.vk_out, a.vk_bstride);
  }
  if (a.wu && a.at_out) {
    dim3 g((unsigned)((a.vocab + kFoldR - 1) / kFoldR), (unsigned)nb);
    if (a.wu_dtype == LOCA_BF16)
      k_head_fold<uint16_t><<<g, kT, 0, st>>>(a.vocab, d, (int)k, (const uint16_t*)a.wu, vk, a.at_out, a.at_bstride);
    else
      k_head_fold<float><<<g, kT, 0, st>>>(a.vocab, d, (int)k, (const float*)a.wu, vk, a.at_out, a.at_bstride);
  }
  *ut_out = ut;
  *vs_out = vs;
  return hipGetLastError();
}

// Workspace of the steps both small-probe forms share (R, the factors, the alignment).
static size_t fit_common_ws(int64_t nb, int64_t d, int64_t np_, int64_t k) {
  const int ns = calib_splits(d);
  const int64_t nch = (np_ + kMaxNp - 1) / kMaxNp;
  size_t s = align256(sizeof(float) * np_ * d);                   // R
  s += align256(sizeof(double) * nch * nb * ns * (2 * k * kMaxNp + kMaxNp * kMaxNp));  // alpha partials
  return s + calib_factor_ws(nb, d, np_, k);
}

size_t feedback_fit_ws(int64_t nb, int64_t d, int64_t np_, int64_t k) {
  const int ns = calib_splits(d);
  size_t s = align256(sizeof(double) * ns * np_ * np_);           // Gamma partials
  s += align256(sizeof(double) * np_ * np_);                      // L
  return s + fit_common_ws(nb, d, np_, k);
}

size_t feedback_fit_primal_ws(int64_t nb, int64_t d, int64_t np_, int64_t k) {
  size_t s = align256(sizeof(double) * d * d);                    // S_E = E E^T
  s += align256(sizeof(double) * d * np_);                        // E in fp64 (right-hand sides)
  s += align256(sizeof(float) * d * np_);                         // R^T = (S_E + beta I)^{-1} E
  s += align256(sizeof(int32_t));                                 // the solve's status
  s += ridge_solve_ws(1, d, np_, 1, LOCA_F64);
  return s + fit_common_ws(nb, d, np_, k);
}

// Steps shared by both small-probe forms, given R (np x d) with F_hat_b = G_b R: the rank-k
// truncation, the credit factors, the alignment diagnostic and the folded head.
static hipError_t fit_tail(const CalibArgs& a, const float* R, char* p) {
  const int64_t d = a.d, np_ = a.np_, k = a.k, nb = a.nb;
  const int ns = calib_splits(d);
  const int64_t nch = (np_ + kMaxNp - 1) / kMaxNp;
  p += align256(sizeof(float) * np_ * d);  // R's own slot (filled by the caller)
  double* apart = (double*)p; p += align256(sizeof(double) * nch * nb * ns * (2 * k * kMaxNp + kMaxNp * kMaxNp));
  double* pP = apart;
  double* pQ = apart + nch * nb * ns * k * kMaxNp;
  double* pG = apart + 2 * nch * nb * ns * k * kMaxNp;
  hipStream_t st = a.stream;
  float *ut = nullptr, *vs = nullptr;
  hipError_t e = launch_calib_factors(a, a.g, a.g_bstride, R, 0, nb, np_, p, &ut, &vs);
  if (e != hipSuccess) return e;
  // P = U_k^T G (U_k^T is k x d: L(c, j) = ut[j * d + c]); Q = (V_k S_k)^T E; ||G||^2 from the
  // diagonal of G^T G; each over column chunks of at most 64 probes
  for (int64_t h = 0; h < nch; ++h) {
    const int64_t c0 = h * kMaxNp;
    const int w = (int)(np_ - c0 < kMaxNp ? np_ - c0 : kMaxNp);
    const dim3 g((unsigned)ns, (unsigned)nb);
    k_tall_cross<float><<<g, kT, 0, st>>>(d, (int)k, w, ut, k * d, 1, d, a.g + c0, a.g_bstride, np_, 1, ns,
                                          pP + h * nb * ns * k * kMaxNp);
    k_tall_cross<float><<<g, kT, 0, st>>>(d, (int)k, w, vs, d * k, k, 1, a.e + c0, 0, np_, 1, ns,
                                          pQ + h * nb * ns * k * kMaxNp);
    k_tall_cross<float><<<g, kT, 0, st>>>(d, w, w, a.g + c0, a.g_bstride, np_, 1, a.g + c0, a.g_bstride, np_, 1, ns,
                                          pG + h * nb * ns * kMaxNp * kMaxNp);
  }
  k_calib_alpha<<<(unsigned)nb, kT, 0, st>>>(nb, (int)k, (int)np_, ns, pP, pQ, pG, a.alpha_out);
  return hipGetLastError();
}

hipError_t launch_feedback_fit(const CalibArgs& a) {
  const int64_t d = a.d, np_ = a.np_, nb = a.nb;
  const int ns = calib_splits(d);
  hipStream_t st = a.stream;
  char* p = a.ws;
  k_zero_i32<<<(unsigned)((nb + 255) / 256), 256, 0, st>>>(a.dev_info, nb);
  if (!a.primal) {
    // dual form: Gamma = E^T E, its Cholesky with beta, R = (Gamma + beta I)^{-1} E^T
    double* gpart = (double*)p; p += align256(sizeof(double) * ns * np_ * np_);
    double* Lmat = (double*)p; p += align256(sizeof(double) * np_ * np_);
    float* R = (float*)p;
    k_tall_cross<float><<<dim3((unsigned)ns, 1), kT, 0, st>>>(d, (int)np_, (int)np_, a.e, 0, np_, 1, a.e, 0, np_, 1,
                                                              ns, gpart);
    k_chol_small<<<1, kT, 0, st>>>((int)np_, ns, gpart, a.beta, Lmat, a.dev_info, nb);
    k_ridge_cols<<<(unsigned)((d + kT - 1) / kT), kT, 0, st>>>(d, (int)np_, a.e, Lmat, R);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return fit_tail(a, R, p);
  }
  // primal form: (E E^T + beta I) R^T = E by the Cholesky solve in d unknowns (np right-hand
  // sides), R = (R^T)^T, so that F_hat_b = G_b E^T (E E^T + beta I)^{-1} = G_b R
  double* SE = (double*)p; p += align256(sizeof(double) * d * d);
  double* E64 = (double*)p; p += align256(sizeof(double) * d * np_);
  float* Rt = (float*)p; p += align256(sizeof(float) * d * np_);
  int32_t* sinfo = (int32_t*)p; p += align256(sizeof(int32_t));
  char* sws = p; p += ridge_solve_ws(1, d, np_, 1, LOCA_F64);
  float* R = (float*)p;
  k_rows_gram<<<dim3((unsigned)((d + 255) / 256), (unsigned)d), 256, 0, st>>>(d, (int)np_, a.e, SE);
  k_to_f64<<<(unsigned)((d * np_ + 255) / 256), 256, 0, st>>>(d * np_, a.e, E64);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const double lam[1] = {a.beta};
  SolveArgs sa{st, 1, d, np_, SE, E64, LOCA_F64, d * d, d * np_, nullptr, nullptr, 0, 0, 0, lam, 1, Rt, d * np_,
               nullptr, 0, nullptr, 0, sinfo, sws};
  if ((e = launch_ridge_solve(sa)) != hipSuccess) return e;
  k_copy_info<<<1, 64, 0, st>>>(sinfo, a.dev_info, nb);
  k_transpose_f32<<<dim3((unsigned)((d + 31) / 32), (unsigned)((np_ + 31) / 32)), 256, 0, st>>>(d, (int)np_, Rt, R);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  return fit_tail(a, R, p);
}

}  // namespace loca
