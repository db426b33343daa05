// k_chol.hip -- ridge solve (row a5 of the step).
//
// Eq. 7 / Theorem S6.1 in the linear-system form of Section S7:
//   (S + lam I) M = [S Lp | K]      (positive definite for lam > 0; no inverse)
// solved for every (block, lam) pair of a call in one batched pass:
//   1. Jacobi equilibration  A^ = D (S + lam I) D,  D = diag(S + lam I)^{-1/2};
//   2. right-looking blocked Cholesky A^ = U^T U (U upper, row-major), panel
//      width 64.  Per panel: one kernel factors the 64 x 64 diagonal block in
//      LDS (every workgroup redundantly, so no extra launch) and applies
//      U11^{-T} to its chunk of the row panel -- the right-hand sides ride
//      along as extra columns, so the forward substitution is free; a second
//      kernel applies the symmetric rank-64 update to the trailing matrix and
//      the right-hand sides with matrix-core MFMA (fp32 32x32x2, or fp64
//      16x16x4 in fp32 mode);
//   3. back substitution U M' = Y by row blocks, M = D M'.
// The first non-positive pivot is reported in dev_info (1-based).
#include "loca_common.h"

namespace loca {

namespace {

constexpr int kP = 64;        // panel width
constexpr int kCW = 64;       // column chunk of the panel kernel
constexpr int kT = 256;       // threads
constexpr int kMC = 16;       // right-hand-side columns per back-substitution workgroup

struct Lams {
  double v[8];
};
__global__ void k_set_lambdas(Lams l, double* out, int cnt) {
  if ((int)threadIdx.x < cnt) out[threadIdx.x] = l.v[threadIdx.x];
}

__global__ void k_fill_zero_i32(int32_t* p, int64_t cnt) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < cnt) p[i] = 0;
}

// D[mi][i] = 1 / sqrt(S_ii + lam_l) for matrix mi = b * nl + l.
template <typename T, typename ST>
__global__ void k_equil_diag(int64_t d, const ST* __restrict__ S, int64_t s_bstride, const double* __restrict__ lam,
                             int nl, T* __restrict__ D) {
  const int64_t mi = blockIdx.y;
  const int64_t b = mi / nl;
  const int l = (int)(mi % nl);
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= d) return;
  const double v = (double)S[b * s_bstride + i * d + i] + lam[l];
  D[mi * d + i] = (T)(1.0 / sqrt(v));
}

// F[i][j] = D_i (S_ij + lam delta_ij) D_j for j >= i; RHS[i][c] = D_i [S Lp | K][i][c].
template <typename T, typename ST>
__global__ void k_equil_setup(int64_t d, int64_t m, int64_t r_prev, const ST* __restrict__ S, int64_t s_bstride,
                              const ST* __restrict__ K, int64_t k_bstride, const double* __restrict__ SLp,
                              const double* __restrict__ lam, int nl, const T* __restrict__ D, T* __restrict__ F,
                              T* __restrict__ R) {
  const int64_t mi = blockIdx.z;
  const int64_t b = mi / nl;
  const int l = (int)(mi % nl);
  const int64_t i = blockIdx.y;
  const T* Dm = D + mi * d;
  const double di = (double)Dm[i];
  const ST* Si = S + b * s_bstride + i * d;
  T* Fi = F + mi * d * d + i * d;
  const int64_t k = m - r_prev;
  for (int64_t j = i + (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j < d; j += (int64_t)gridDim.x * blockDim.x) {
    const double v = (double)Si[j] + (j == i ? lam[l] : 0.0);
    Fi[j] = (T)(di * v * (double)Dm[j]);
  }
  if (blockIdx.x == 0)
    for (int64_t c = threadIdx.x; c < m; c += blockDim.x) {
      double v = (c < r_prev) ? SLp[b * d * r_prev + i * r_prev + c] : (double)K[b * k_bstride + i * k + (c - r_prev)];
      R[mi * d * m + i * m + c] = (T)(di * v);
    }
}

// SLp[b] = S_sym Lp (d x r_prev, fp64) from the upper triangle of S.
template <typename ST>
__global__ void k_sym_mul(int64_t d, int64_t r_prev, const ST* __restrict__ S, int64_t s_bstride,
                          const float* __restrict__ Lp, int64_t lp_bstride, double* __restrict__ out) {
  const int64_t b = blockIdx.y;
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= d * r_prev) return;
  const int64_t i = e / r_prev, c = e % r_prev;
  const ST* Sb = S + b * s_bstride;
  const float* L = Lp + b * lp_bstride;
  double s = 0.0;
  for (int64_t j = 0; j < d; ++j) {
    const double sij = (j >= i) ? (double)Sb[i * d + j] : (double)Sb[j * d + i];
    s += sij * (double)L[j * r_prev + c];
  }
  out[b * d * r_prev + e] = s;
}

// ------------------------------------------------------------------ panel: factor U11, apply U11^{-T}

// U11 of panel p is written to Ud (nm x d x kP): the workgroups of this launch still read the
// unfactored block from F, so it must not be overwritten in place.
template <typename T>
__global__ __launch_bounds__(kT) void k_chol_panel(int64_t d, int64_t m, int64_t p, T* __restrict__ Fall,
                                                   T* __restrict__ Rall, T* __restrict__ Udall,
                                                   int32_t* __restrict__ dev_info) {
  __shared__ T sU[kP][kP + 1];
  __shared__ T sX[kP][kCW + 1];
  const int64_t mi = blockIdx.y;
  T* F = Fall + mi * d * d;
  T* R = Rall + mi * d * m;
  const int pw = (int)((d - p) < kP ? (d - p) : kP);
  const int tid = threadIdx.x;
  for (int e = tid; e < kP * kP; e += kT) {
    const int r = e / kP, c = e % kP;
    sU[r][c] = (r < pw && c < pw && c >= r) ? F[(p + r) * d + p + c] : (T)0;
  }
  __syncthreads();
  // unblocked right-looking Cholesky of the diagonal block (upper factor)
  for (int j = 0; j < pw; ++j) {
    const T piv = sU[j][j];
    if (!(piv > (T)0) && tid == 0 && blockIdx.x == 0) atomicCAS(&dev_info[mi], 0, (int32_t)(p + j + 1));
    const T ujj = sqrt(piv);
    __syncthreads();
    for (int c = j + tid; c < pw; c += kT) sU[j][c] = (c == j) ? ujj : sU[j][c] / ujj;
    __syncthreads();
    const int rem = pw - j - 1;
    for (int e = tid; e < rem * rem; e += kT) {
      const int r = j + 1 + e / rem, c = j + 1 + e % rem;
      if (c >= r) sU[r][c] -= sU[j][r] * sU[j][c];
    }
    __syncthreads();
  }
  if (blockIdx.x == 0) {
    T* Ud = Udall + mi * d * kP + p * kP;  // rows p..p+pw, kP columns
    for (int e = tid; e < kP * kP; e += kT) {
      const int r = e / kP, c = e % kP;
      if (r < pw) Ud[r * kP + c] = (c >= r && c < pw) ? sU[r][c] : (T)0;
    }
  }
  // this workgroup's chunk: columns of F right of the block, then the RHS columns
  const int64_t nrem = d - p - pw;
  const int64_t nchF = (nrem + kCW - 1) / kCW;
  const bool rhs = (int64_t)blockIdx.x >= nchF;
  const int64_t c0 = rhs ? ((int64_t)blockIdx.x - nchF) * kCW : p + pw + (int64_t)blockIdx.x * kCW;
  const int64_t cend = rhs ? m : d;
  if (c0 >= cend) return;
  const int cw = (int)((cend - c0) < kCW ? (cend - c0) : kCW);
  for (int e = tid; e < kP * kCW; e += kT) {
    const int r = e / kCW, c = e % kCW;
    T v = (T)0;
    if (r < pw && c < cw) v = rhs ? R[(p + r) * m + c0 + c] : F[(p + r) * d + c0 + c];
    sX[r][c] = v;
  }
  __syncthreads();
  // forward substitution U11^T X = A (U11^T lower): row r final, then eliminate below
  for (int r = 0; r < pw; ++r) {
    for (int c = tid; c < cw; c += kT) sX[r][c] /= sU[r][r];
    __syncthreads();
    const int rem = pw - r - 1;
    for (int e = tid; e < rem * cw; e += kT) {
      const int s = r + 1 + e / cw, c = e % cw;
      sX[s][c] -= sU[r][s] * sX[r][c];
    }
    __syncthreads();
  }
  for (int e = tid; e < pw * cw; e += kT) {
    const int r = e / cw, c = e % cw;
    if (rhs) R[(p + r) * m + c0 + c] = sX[r][c];
    else F[(p + r) * d + c0 + c] = sX[r][c];
  }
}

// ------------------------------------------------------------------ trailing update (fp32 MFMA)

// Jobs: upper 128 x 128 tiles of the trailing matrix, then 128 x 128 tiles of the RHS rows.
// Out -= Panel^T Q with Panel = rows [p, p+pw) of F (columns of the tile's rows) and
// Q = the same rows of F (tile's columns) or of R.
constexpr int kUT = 128;

LOCA_DEV void upper_tile_c(int u, int T, int& I, int& J) {
  int i = 0;
  while (u >= T - i) { u -= T - i; ++i; }
  I = i;
  J = i + u;
}

__global__ __launch_bounds__(kT) void k_chol_update_f32(int64_t d, int64_t m, int64_t p, float* __restrict__ Fall,
                                                        float* __restrict__ Rall) {
  __shared__ float sP[kP][kUT + 4];
  __shared__ float sQ[kP][kUT + 4];
  const int64_t mi = blockIdx.y;
  float* F = Fall + mi * d * d;
  float* R = Rall + mi * d * m;
  const int pw = (int)((d - p) < kP ? (d - p) : kP);
  const int64_t off = p + pw, nrem = d - off;
  const int T2 = (int)((nrem + kUT - 1) / kUT);
  const int nU = T2 * (T2 + 1) / 2;
  const int TM = (int)((m + kUT - 1) / kUT);
  int I, J;
  bool rhs = (int)blockIdx.x >= nU;
  if (!rhs) upper_tile_c(blockIdx.x, T2, I, J);
  else { const int u = blockIdx.x - nU; I = u / TM; J = u % TM; }
  const int64_t r0 = off + (int64_t)I * kUT;                 // output rows (and panel columns)
  const int64_t c0 = rhs ? (int64_t)J * kUT : off + (int64_t)J * kUT;
  const int64_t cend = rhs ? m : d;
  const int tid = threadIdx.x;
  for (int e = tid; e < kP * kUT; e += kT) {
    const int kk = e / kUT, c = e % kUT;
    float a = 0.f, q = 0.f;
    if (kk < pw) {
      if (r0 + c < d) a = F[(p + kk) * d + r0 + c];
      if (c0 + c < cend) q = rhs ? R[(p + kk) * m + c0 + c] : F[(p + kk) * d + c0 + c];
    }
    sP[kk][c] = a;
    sQ[kk][c] = q;
  }
  __syncthreads();
  const int lane = tid & 63, wid = tid >> 6, wi = wid >> 1, wj = wid & 1;
  if (!rhs && I == J && wi > wj) return;  // strictly lower quarter of a diagonal tile
  f32x16_t acc[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.f;
  for (int kk = 0; kk < kP; kk += 2) {
    float fa[2], fb[2];
#pragma unroll
    for (int a = 0; a < 2; ++a) fa[a] = sP[kk + (lane >> 5)][wi * 64 + 32 * a + (lane & 31)];
#pragma unroll
    for (int b = 0; b < 2; ++b) fb[b] = sQ[kk + (lane >> 5)][wj * 64 + 32 * b + (lane & 31)];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
      for (int b = 0; b < 2; ++b) acc[a][b] = mfma_f32x2(fa[a], fb[b], acc[a][b]);
  }
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t row = r0 + wi * 64 + 32 * a + mfma32_row(lane, r);
        const int64_t col = c0 + wj * 64 + 32 * b + mfma32_col(lane);
        if (row < d && col < cend) {
          if (rhs) R[row * m + col] -= acc[a][b][r];
          else if (col >= row) F[row * d + col] -= acc[a][b][r];
        }
      }
}

// fp64 variant: 64 x 64 tiles, 4 waves of 32 x 32 (2 x 2 blocks of 16 x 16).
constexpr int kUT64 = 64;

__global__ __launch_bounds__(kT) void k_chol_update_f64(int64_t d, int64_t m, int64_t p, double* __restrict__ Fall,
                                                        double* __restrict__ Rall) {
  __shared__ double sP[kP][kUT64 + 1];
  __shared__ double sQ[kP][kUT64 + 1];
  const int64_t mi = blockIdx.y;
  double* F = Fall + mi * d * d;
  double* R = Rall + mi * d * m;
  const int pw = (int)((d - p) < kP ? (d - p) : kP);
  const int64_t off = p + pw, nrem = d - off;
  const int T2 = (int)((nrem + kUT64 - 1) / kUT64);
  const int nU = T2 * (T2 + 1) / 2;
  const int TM = (int)((m + kUT64 - 1) / kUT64);
  int I, J;
  bool rhs = (int)blockIdx.x >= nU;
  if (!rhs) upper_tile_c(blockIdx.x, T2, I, J);
  else { const int u = blockIdx.x - nU; I = u / TM; J = u % TM; }
  const int64_t r0 = off + (int64_t)I * kUT64;
  const int64_t c0 = rhs ? (int64_t)J * kUT64 : off + (int64_t)J * kUT64;
  const int64_t cend = rhs ? m : d;
  const int tid = threadIdx.x;
  for (int e = tid; e < kP * kUT64; e += kT) {
    const int kk = e / kUT64, c = e % kUT64;
    double a = 0.0, q = 0.0;
    if (kk < pw) {
      if (r0 + c < d) a = F[(p + kk) * d + r0 + c];
      if (c0 + c < cend) q = rhs ? R[(p + kk) * m + c0 + c] : F[(p + kk) * d + c0 + c];
    }
    sP[kk][c] = a;
    sQ[kk][c] = q;
  }
  __syncthreads();
  const int lane = tid & 63, wid = tid >> 6, wi = wid >> 1, wj = wid & 1;
  f64x4_t acc[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) acc[a][b] = (f64x4_t){0.0, 0.0, 0.0, 0.0};
  for (int kk = 0; kk < kP; kk += 4) {
    double fa[2], fb[2];
#pragma unroll
    for (int a = 0; a < 2; ++a) fa[a] = sP[kk + (lane >> 4)][wi * 32 + 16 * a + (lane & 15)];
#pragma unroll
    for (int b = 0; b < 2; ++b) fb[b] = sQ[kk + (lane >> 4)][wj * 32 + 16 * b + (lane & 15)];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
      for (int b = 0; b < 2; ++b) acc[a][b] = mfma_f64(fa[a], fb[b], acc[a][b]);
  }
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t row = r0 + wi * 32 + 16 * a + (lane >> 4) + 4 * r;
        const int64_t col = c0 + wj * 32 + 16 * b + (lane & 15);
        if (row < d && col < cend) {
          if (rhs) R[row * m + col] -= acc[a][b][r];
          else if (col >= row) F[row * d + col] -= acc[a][b][r];
        }
      }
}

// ------------------------------------------------------------------ back substitution U M' = Y, M = D M'

template <typename T>
__global__ __launch_bounds__(kT) void k_chol_backsolve(int64_t d, int64_t m, const T* __restrict__ Fall,
                                                       const T* __restrict__ Udall, T* __restrict__ Rall,
                                                       const T* __restrict__ Dall, float* __restrict__ Mout,
                                                       int64_t m_bstride) {
  __shared__ T sU[kP][kP + 1];
  __shared__ T sX[kP][kMC + 1];
  __shared__ T sAcc[kP][kMC + 1];
  const int64_t mi = blockIdx.y;
  const T* F = Fall + mi * d * d;
  T* R = Rall + mi * d * m;
  const int64_t c0 = (int64_t)blockIdx.x * kMC;
  const int mc = (int)((m - c0) < kMC ? (m - c0) : kMC);
  const int tid = threadIdx.x;
  const int64_t nblk = (d + kP - 1) / kP;
  for (int64_t pb = nblk - 1; pb >= 0; --pb) {
    const int64_t p0 = pb * kP;
    const int pw = (int)((d - p0) < kP ? (d - p0) : kP);
    const int64_t p1 = p0 + pw;
    // acc = sum_{j >= p1} U[p0 + r][j] M'[j][c]; each thread owns (r, c) pairs e = tid + 256 q
    T acc[(kP * kMC) / kT];
#pragma unroll
    for (int q = 0; q < (kP * kMC) / kT; ++q) acc[q] = (T)0;
    for (int64_t j0 = p1; j0 < d; j0 += kP) {
      const int jw = (int)((d - j0) < kP ? (d - j0) : kP);
      __syncthreads();
      for (int e = tid; e < kP * kP; e += kT) {
        const int r = e / kP, jj = e % kP;
        sU[r][jj] = (r < pw && jj < jw) ? F[(p0 + r) * d + j0 + jj] : (T)0;
      }
      for (int e = tid; e < kP * kMC; e += kT) {
        const int jj = e / kMC, c = e % kMC;
        sX[jj][c] = (jj < jw && c < mc) ? R[(j0 + jj) * m + c0 + c] : (T)0;
      }
      __syncthreads();
#pragma unroll
      for (int q = 0; q < (kP * kMC) / kT; ++q) {
        const int e = tid + kT * q;
        const int r = e / kMC, c = e % kMC;
        T s = acc[q];
        for (int jj = 0; jj < kP; ++jj) s += sU[r][jj] * sX[jj][c];
        acc[q] = s;
      }
    }
    __syncthreads();
    for (int e = tid; e < kP * kP; e += kT) {
      const int r = e / kP, c = e % kP;
      sU[r][c] = (r < pw && c < pw) ? Udall[mi * d * kP + (p0 + r) * kP + c] : (T)0;
    }
#pragma unroll
    for (int q = 0; q < (kP * kMC) / kT; ++q) {
      const int e = tid + kT * q;
      const int r = e / kMC, c = e % kMC;
      sAcc[r][c] = (r < pw && c < mc) ? R[(p0 + r) * m + c0 + c] - acc[q] : (T)0;
    }
    __syncthreads();
    for (int r = pw - 1; r >= 0; --r) {
      if (tid < mc) sAcc[r][tid] /= sU[r][r];
      __syncthreads();
      for (int e = tid; e < r * mc; e += kT) {
        const int s = e / mc, c = e % mc;
        sAcc[s][c] -= sU[s][r] * sAcc[r][c];
      }
      __syncthreads();
    }
    for (int e = tid; e < pw * mc; e += kT) {
      const int r = e / mc, c = e % mc;
      R[(p0 + r) * m + c0 + c] = sAcc[r][c];
    }
  }
  __syncthreads();
  const T* D = Dall + mi * d;
  float* M = Mout + mi * m_bstride;
  for (int64_t e = tid; e < d * mc; e += kT) {
    const int64_t i = e / mc;
    const int c = (int)(e % mc);
    M[i * m + c0 + c] = (float)(D[i] * R[i * m + c0 + c]);
  }
}

template <typename T>
size_t solve_ws_t(int64_t nb, int64_t d, int64_t m, int64_t nl, int64_t r_prev) {
  const int64_t nm = nb * nl;
  size_t s = align256(sizeof(T) * nm * d * d);  // F
  s += align256(sizeof(T) * nm * d * m);         // R
  s += align256(sizeof(T) * nm * d);             // D
  s += align256(sizeof(double) * nb * d * (r_prev > 0 ? r_prev : 1));  // S Lp
  s += 256;                                                            // lambdas
  s += align256(sizeof(T) * nm * d * kP);                              // diagonal blocks U11
  return s;
}

template <typename T, typename ST>
hipError_t run_solve(const SolveArgs& a) {
  const int64_t d = a.d, m = a.r_prev + a.k, nl = a.n_lambda, nm = a.nb * nl;
  char* p = a.ws;
  T* F = (T*)p; p += align256(sizeof(T) * nm * d * d);
  T* R = (T*)p; p += align256(sizeof(T) * nm * d * m);
  T* D = (T*)p; p += align256(sizeof(T) * nm * d);
  double* SLp = (double*)p;
  Lams lams;
  for (int i = 0; i < 8; ++i) lams.v[i] = (i < nl) ? a.lambdas[i] : 0.0;
  double* dlam = (double*)(p + align256(sizeof(double) * a.nb * d * (a.r_prev > 0 ? a.r_prev : 1)));
  T* Ud = (T*)((char*)dlam + 256);
  // the host lambdas travel by value into a one-wave kernel (no copy from pageable memory)
  k_set_lambdas<<<1, 64, 0, a.stream>>>(lams, dlam, (int)nl);
  k_fill_zero_i32<<<(unsigned)((nm + 255) / 256), 256, 0, a.stream>>>(a.dev_info, nm);
  const ST* S = (const ST*)a.S;
  const ST* K = (const ST*)a.K;
  if (a.r_prev > 0) {
    dim3 g((unsigned)((d * a.r_prev + 255) / 256), (unsigned)a.nb);
    k_sym_mul<ST><<<g, 256, 0, a.stream>>>(d, a.r_prev, S, a.s_bstride, a.lp, a.lp_bstride, SLp);
  }
  {
    dim3 g((unsigned)((d + 255) / 256), (unsigned)nm);
    k_equil_diag<T, ST><<<g, 256, 0, a.stream>>>(d, S, a.s_bstride, dlam, (int)nl, D);
    dim3 g2((unsigned)((d + 255) / 256 < 8 ? (d + 255) / 256 : 8), (unsigned)d, (unsigned)nm);
    k_equil_setup<T, ST><<<g2, 256, 0, a.stream>>>(d, m, a.r_prev, S, a.s_bstride, K, a.k_bstride, SLp, dlam,
                                                   (int)nl, D, F, R);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  for (int64_t pp = 0; pp < d; pp += kP) {
    const int64_t pw = (d - pp) < kP ? (d - pp) : kP;
    const int64_t nrem = d - pp - pw;
    const int64_t nch = (nrem + kCW - 1) / kCW + (m + kCW - 1) / kCW;
    k_chol_panel<T><<<dim3((unsigned)nch, (unsigned)nm), kT, 0, a.stream>>>(d, m, pp, F, R, Ud, a.dev_info);
    if (nrem > 0) {
      const int64_t ut = sizeof(T) == 4 ? kUT : kUT64;
      const int64_t T2 = (nrem + ut - 1) / ut;
      const int64_t jobs = T2 * (T2 + 1) / 2 + T2 * ((m + ut - 1) / ut);
      if (sizeof(T) == 4)
        k_chol_update_f32<<<dim3((unsigned)jobs, (unsigned)nm), kT, 0, a.stream>>>(d, m, pp, (float*)F, (float*)R);
      else
        k_chol_update_f64<<<dim3((unsigned)jobs, (unsigned)nm), kT, 0, a.stream>>>(d, m, pp, (double*)F, (double*)R);
    }
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  k_chol_backsolve<T><<<dim3((unsigned)((m + kMC - 1) / kMC), (unsigned)nm), kT, 0, a.stream>>>(d, m, F, Ud, R, D, a.m_out,
                                                                                                a.m_bstride);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (a.w_dense_out) {
    // W = M [Rp; B~]: rows of the right factor come from Rp (first r_prev) then B~.
    if (a.r_prev == 0)
      return launch_lowrank_product(a.stream, nm, d, d, m, a.m_out, a.m_bstride, m, a.credit_b, a.b_bstride, nl, d,
                                    a.w_dense_out, a.w_bstride);
    return hipErrorNotSupported;
  }
  return hipSuccess;
}

}  // namespace

size_t ridge_solve_ws(int64_t nb, int64_t d, int64_t m, int64_t n_lambda, loca_dtype acc) {
  // m counts r_prev + k; the S Lp scratch is sized for m columns (>= r_prev)
  size_t s = acc == LOCA_F64 ? solve_ws_t<double>(nb, d, m, n_lambda, m) : solve_ws_t<float>(nb, d, m, n_lambda, m);
  return s;
}

hipError_t launch_ridge_solve(const SolveArgs& a) {
  if (a.acc == LOCA_F64) return run_solve<double, double>(a);
  return run_solve<float, float>(a);
}

}  // namespace loca
