// k_chol.hip -- ridge solve (row a5 of the step).
//
// Eq. 7 / Theorem S6.1 in the linear-system form of Section S7:
//   (S + lam I) M = [S Lp | K]      (positive definite for lam > 0; no inverse)
// solved for every (block, lam) pair of a call in one batched pass:
//   1. Jacobi equilibration  A^ = D (S + lam I) D,  D = diag(S + lam I)^{-1/2};
//   2. right-looking blocked Cholesky A^ = U^T U (U upper, row-major) with
//      P-wide panels (P = 128 in fp32, 64 in fp64).  Per panel, three launches
//      batched over all matrices: the diagonal block is factored and inverted
//      in LDS by one workgroup per matrix; the row panel U12 = U11^{-T} A12 is
//      a matrix-core product with that inverse; the trailing matrix takes the
//      symmetric rank-P update A22 -= U12^T U12.  The right-hand sides ride
//      along as extra columns of the row panel and the update, so the forward
//      substitution costs nothing extra.  Products use MFMA (fp32 32x32x2, or
//      fp64 16x16x4 for fp64 statistics);
//   3. back substitution U M' = Y by row blocks, each a product with U11^{-1},
//      then M = D M'.
// The first non-positive pivot is reported in dev_info (1-based).
#include <mutex>

#include "loca_launch.h"
#include "loca_bf16.h"

#include <functional>
#include <vector>

namespace loca {

namespace {

constexpr int kT = 256;       // threads

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
// One workgroup per (kEqRows rows, block): a row of S is read once for all nl lambdas.
constexpr int kEqRows = 16;
template <typename T, typename ST>
__global__ __launch_bounds__(256) void k_equil_setup(int64_t d, int64_t m, int64_t r_prev, const ST* __restrict__ S,
                                                     int64_t s_bstride, const ST* __restrict__ K, int64_t k_bstride,
                                                     const double* __restrict__ SLp, const double* __restrict__ lam,
                                                     int nl, const T* __restrict__ D, T* __restrict__ F,
                                                     T* __restrict__ R) {
  const int64_t b = blockIdx.y;
  const int64_t k = m - r_prev;
  for (int ii = 0; ii < kEqRows; ++ii) {
    const int64_t i = (int64_t)blockIdx.x * kEqRows + ii;
    if (i >= d) return;
    const ST* Si = S + b * s_bstride + i * d;
    for (int64_t j = i + threadIdx.x; j < d; j += blockDim.x) {
      const double sij = (double)Si[j];
      for (int l = 0; l < nl; ++l) {
        const int64_t mi = b * nl + l;
        const double v = sij + (j == i ? lam[l] : 0.0);
        F[mi * d * d + i * d + j] = (T)((double)D[mi * d + i] * v * (double)D[mi * d + j]);
      }
    }
    for (int64_t c = threadIdx.x; c < m; c += blockDim.x) {
      const double v = (c < r_prev) ? SLp[b * d * r_prev + i * r_prev + c] : (double)K[b * k_bstride + i * k + (c - r_prev)];
      for (int l = 0; l < nl; ++l) {
        const int64_t mi = b * nl + l;
        R[mi * d * m + i * m + c] = (T)((double)D[mi * d + i] * v);
      }
    }
  }
}

// RHS[i][c] = D_i [S Lp | K][i][c] only (the factor of an earlier call is reused).
template <typename T, typename ST>
__global__ void k_equil_rhs(int64_t d, int64_t m, int64_t r_prev, const ST* __restrict__ K, int64_t k_bstride,
                            const double* __restrict__ SLp, int nl, const T* __restrict__ D, T* __restrict__ R) {
  const int64_t mi = blockIdx.y, b = mi / nl;
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= d * m) return;
  const int64_t i = e / m, c = e % m, k = m - r_prev;
  const double v = (c < r_prev) ? SLp[b * d * r_prev + i * r_prev + c] : (double)K[b * k_bstride + i * k + (c - r_prev)];
  R[mi * d * m + e] = (T)((double)D[mi * d + i] * v);
}

// The same for float statistics and factors when d % 4 == 0 and the rows of S are 16-byte
// aligned, tiled so that every workgroup has the same amount of work: a workgroup takes
// kEqRows rows and one chunk of kEqCols columns (chunks wholly below the diagonal exit),
// each thread four consecutive columns (16-byte loads and stores of S, D and F, one load
// of S for all lambdas); the four-column group that holds the diagonal writes only its
// entries on or above it.  The right-hand sides are written by the workgroups of the last
// chunk (never wholly below the diagonal).
// The arithmetic is that of k_equil_setup, term for term.
constexpr int kEqCols = 1024;
__global__ __launch_bounds__(256) void k_equil_setup_v4(int64_t d, int64_t m, int64_t r_prev,
                                                        const float* __restrict__ S, int64_t s_bstride,
                                                        const float* __restrict__ K, int64_t k_bstride,
                                                        const double* __restrict__ SLp,
                                                        const double* __restrict__ lam, int nl,
                                                        const float* __restrict__ D, float* __restrict__ F,
                                                        float* __restrict__ R) {
  const int64_t b = blockIdx.z;
  const int64_t k = m - r_prev;
  const int64_t i0 = (int64_t)blockIdx.x * kEqRows;
  const int64_t c0 = (int64_t)blockIdx.y * kEqCols;
  if (c0 + kEqCols <= (i0 & ~(int64_t)3)) return;  // every row of the tile starts past this chunk
  const int64_t j = c0 + 4 * threadIdx.x;
  const bool jin = j < d;
  // every global load of the tile is issued before the first use: the rows of S at this
  // thread's four columns; per lambda, D at the columns and at the tile's rows
  float4 sv[kEqRows];
#pragma unroll
  for (int ii = 0; ii < kEqRows; ++ii) {
    const int64_t i = i0 + ii;
    const bool need = jin && i < d && j + 3 >= i;
    sv[ii] = *(const float4*)(S + b * s_bstride + (need ? i * d + j : 0));
  }
  for (int l = 0; l < nl; ++l) {
    const int64_t mi = b * nl + l;
    const float4 dj = *(const float4*)(D + mi * d + (jin ? j : 0));
    float di[kEqRows];
#pragma unroll
    for (int ii = 0; ii < kEqRows; ++ii) di[ii] = D[mi * d + (i0 + ii < d ? i0 + ii : d - 1)];
    const double li = lam[l];
#pragma unroll
    for (int ii = 0; ii < kEqRows; ++ii) {
      const int64_t i = i0 + ii;
      if (i < d && jin && j + 3 >= i) {
        const double dd = (double)di[ii];
        float o[4];
        o[0] = (float)(dd * ((double)sv[ii].x + (j == i ? li : 0.0)) * (double)dj.x);
        o[1] = (float)(dd * ((double)sv[ii].y + (j + 1 == i ? li : 0.0)) * (double)dj.y);
        o[2] = (float)(dd * ((double)sv[ii].z + (j + 2 == i ? li : 0.0)) * (double)dj.z);
        o[3] = (float)(dd * ((double)sv[ii].w + (j + 3 == i ? li : 0.0)) * (double)dj.w);
        float* dst = F + mi * d * d + i * d + j;
        if (j >= i) {
          *(float4*)dst = make_float4(o[0], o[1], o[2], o[3]);
        } else {
#pragma unroll
          for (int u = 1; u < 4; ++u)
            if (j + u >= i) dst[u] = o[u];
        }
      }
    }
  }
  if (blockIdx.y == gridDim.y - 1)  // the last chunk holds column d - 1 >= i of every row
    for (int ii = 0; ii < kEqRows; ++ii) {
      const int64_t i = i0 + ii;
      if (i >= d) break;
      for (int64_t c = threadIdx.x; c < m; c += blockDim.x) {
        const double v = (c < r_prev) ? SLp[b * d * r_prev + i * r_prev + c] : (double)K[b * k_bstride + i * k + (c - r_prev)];
        for (int l = 0; l < nl; ++l) {
          const int64_t mi = b * nl + l;
          R[mi * d * m + i * m + c] = (float)((double)D[mi * d + i] * v);
        }
      }
    }
}

// SLp[b] = S_sym Lp (d x r_prev, fp64) from the upper triangle of S.  A workgroup owns 64
// rows and RC columns of the product (grid: x over row tiles, y = block, z over column
// chunks) and walks the 64-wide column tiles of S in order: tiles on or above the
// diagonal are read row-major, tiles below it as the transpose of the stored tile above
// (both with coalesced rows), the diagonal tile mirrored from its upper half.  Thread t
// owns row t % 64 and all RC columns; wave q = t / 64 takes the columns 16q .. 16q + 15 of
// each tile, and the four waves' sums are added in a fixed order at the end.
constexpr int kSM = 64;
template <typename ST, int RC>
__global__ __launch_bounds__(256) void k_sym_mul(int64_t d, int64_t r_prev, const ST* __restrict__ S,
                                                 int64_t s_bstride, const float* __restrict__ Lp,
                                                 int64_t lp_bstride, double* __restrict__ out) {
  __shared__ ST sS[kSM][kSM + 1];
  __shared__ __attribute__((aligned(16))) float sL[kSM][RC];
  __shared__ double sR[3][kSM][RC + 1];
  const int64_t b = blockIdx.y;
  const int64_t i0 = (int64_t)blockIdx.x * kSM;
  const int64_t c0 = (int64_t)blockIdx.z * RC;
  const ST* Sb = S + b * s_bstride;
  const float* L = Lp + b * lp_bstride;
  const int t = threadIdx.x, r = t & 63, q = t >> 6;
  double acc[RC];
#pragma unroll
  for (int u = 0; u < RC; ++u) acc[u] = 0.0;
  for (int64_t j0 = 0; j0 < d; j0 += kSM) {
    __syncthreads();
    // sS[rr][cc] = S_sym[i0 + rr][j0 + cc]
    for (int e = t; e < kSM * kSM; e += 256) {
      const int rr = e / kSM, cc = e % kSM;
      if (j0 >= i0) {  // rows i0 + rr, columns j0 + cc (the diagonal tile is fixed up below)
        const int64_t gi = i0 + rr, gj = j0 + cc;
        sS[rr][cc] = (gi < d && gj < d) ? Sb[gi * d + gj] : (ST)0;
      } else {         // stored tile (j0, i0): rows j0 + rr, columns i0 + cc, transposed
        const int64_t gi = j0 + rr, gj = i0 + cc;
        sS[cc][rr] = (gi < d && gj < d) ? Sb[gi * d + gj] : (ST)0;
      }
    }
    for (int e = t; e < kSM * RC; e += 256) {
      const int rr = e / RC, cc = e % RC;
      sL[rr][cc] = (j0 + rr < d && c0 + cc < r_prev) ? L[(j0 + rr) * r_prev + c0 + cc] : 0.f;
    }
    __syncthreads();
    if (j0 == i0) {  // mirror the upper half of the diagonal tile
      for (int e = t; e < kSM * kSM; e += 256) {
        const int rr = e / kSM, cc = e % kSM;
        if (cc < rr) sS[rr][cc] = sS[cc][rr];
      }
      __syncthreads();
    }
#pragma unroll 4
    for (int jj = 16 * q; jj < 16 * q + 16; ++jj) {
      const double sv = (double)sS[r][jj];
#pragma unroll
      for (int u = 0; u < RC; u += 4) {
        const float4 l = *(const float4*)&sL[jj][u];
        acc[u] += sv * (double)l.x;
        acc[u + 1] += sv * (double)l.y;
        acc[u + 2] += sv * (double)l.z;
        acc[u + 3] += sv * (double)l.w;
      }
    }
  }
  if (q > 0)
#pragma unroll
    for (int u = 0; u < RC; ++u) sR[q - 1][r][u] = acc[u];
  __syncthreads();
  if (q == 0 && i0 + r < d)
#pragma unroll
    for (int u = 0; u < RC; ++u) {
      const double v = ((acc[u] + sR[0][r][u]) + sR[1][r][u]) + sR[2][r][u];
      if (c0 + u < r_prev) out[b * d * r_prev + (i0 + r) * r_prev + c0 + u] = v;
    }
}

// ------------------------------------------------------------------ matrix-core tile products

// Per precision: panel width P (= output tile side), MFMA block side BLK and its K step.
template <typename T> struct Mf;
template <> struct Mf<float> {
  static constexpr int P = 128, BLK = 32, KS = 2, NR = 16;
  typedef f32x16_t acc_t;
  static LOCA_DEV acc_t mma(float a, float b, acc_t c) { return mfma_f32x2(a, b, c); }
  static LOCA_DEV int row(int lane, int r) { return mfma32_row(lane, r); }
  static LOCA_DEV int col(int lane) { return lane & 31; }
  static LOCA_DEV acc_t zero() { acc_t z; for (int r = 0; r < 16; ++r) z[r] = 0.f; return z; }
};
template <> struct Mf<double> {
  static constexpr int P = 64, BLK = 16, KS = 4, NR = 4;
  typedef f64x4_t acc_t;
  static LOCA_DEV acc_t mma(double a, double b, acc_t c) { return mfma_f64(a, b, c); }
  static LOCA_DEV int row(int lane, int r) { return (lane >> 4) + 4 * r; }
  static LOCA_DEV int col(int lane) { return lane & 15; }
  static LOCA_DEV acc_t zero() { return (acc_t){0.0, 0.0, 0.0, 0.0}; }
};

// acc[m][q] += sum_kk sP[kk][i] sQ[kk][j] over the wave's (P/2) x (P/2) quarter (wi, wj) of a
// P x P output tile; sP, sQ are K x (P + pad) row-major LDS panels.
template <typename T>
LOCA_DEV void tile_mma(const T* sP, const T* sQ, int ld, int K, int wi, int wj, int lane,
                       typename Mf<T>::acc_t (&acc)[2][2]) {
  constexpr int BLK = Mf<T>::BLK, KS = Mf<T>::KS, WT = Mf<T>::P / 2;
  const int kr = lane / BLK, cr = lane % BLK;
  for (int kk = 0; kk < K; kk += KS) {
    T a[2], b[2];
#pragma unroll
    for (int m = 0; m < 2; ++m) a[m] = sP[(kk + kr) * ld + wi * WT + m * BLK + cr];
#pragma unroll
    for (int q = 0; q < 2; ++q) b[q] = sQ[(kk + kr) * ld + wj * WT + q * BLK + cr];
#pragma unroll
    for (int m = 0; m < 2; ++m)
#pragma unroll
      for (int q = 0; q < 2; ++q) acc[m][q] = Mf<T>::mma(a[m], b[q], acc[m][q]);
  }
}

// ------------------------------------------------------------------ diagonal block: factor and invert

// One workgroup per matrix factors the P x P diagonal block, A11 = U11^T U11, and
// inverts U11.  The block lives in registers: thread (ty, tx) of a 16 x 16 grid owns
// the entries (ty + 16 i, tx + 16 k).  Step j of the factorization needs only row j,
// which its owners publish to a double-buffered LDS row, so each step costs one
// barrier.  The inverse X = U11^{-1} is built bottom-up the same way (row i of X is
// final once rows > i have been applied).  X replaces the diagonal block of F (strict
// lower part zeroed): the row panel and the back substitution apply it as a product.
template <typename T>
__global__ __launch_bounds__(kT) void k_diag_block(int64_t d, int64_t p, T* __restrict__ Fall,
                                                   int32_t* __restrict__ dev_info) {
  constexpr int P = Mf<T>::P, NI = P / 16;
  __shared__ T rowbuf[2][P];
  __shared__ T sU[P][P + 1];
  const int64_t mi = blockIdx.x;
  T* F = Fall + mi * d * d;
  const T* A0 = F + p * d + p;
  const int pw = (int)((d - p) < P ? (d - p) : P);
  const int tid = threadIdx.x, ty = tid >> 4, tx = tid & 15;
  T a[NI][NI];
#pragma unroll
  for (int i = 0; i < NI; ++i)
#pragma unroll
    for (int k = 0; k < NI; ++k) {
      const int r = ty + 16 * i, c = tx + 16 * k;
      a[i][k] = ld_or_zero(A0, (int64_t)r * d + c, r < pw && c < pw && c >= r);
    }
  if (ty == 0)
#pragma unroll
    for (int k = 0; k < NI; ++k) rowbuf[0][tx + 16 * k] = a[0][k];
  for (int j = 0; j < pw; ++j) {
    __syncthreads();
    const T* rb = rowbuf[j & 1];
    const T piv = rb[j];
    if (!(piv > (T)0) && tid == 0) atomicCAS(&dev_info[mi], 0, (int32_t)(p + j + 1));
    const T ujj = sqrt(piv);
    const T inv = (T)1 / ujj;
    T ur[NI], uc[NI];
#pragma unroll
    for (int i = 0; i < NI; ++i) ur[i] = rb[ty + 16 * i] * inv;
#pragma unroll
    for (int k = 0; k < NI; ++k) uc[k] = rb[tx + 16 * k] * inv;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int r = ty + 16 * i;
      if (r == j) {  // owners of row j: final row of U
#pragma unroll
        for (int k = 0; k < NI; ++k) {
          const int c = tx + 16 * k;
          if (c >= j && c < pw) a[i][k] = (c == j) ? ujj : uc[k];
        }
      } else if (r > j && r < pw) {
#pragma unroll
        for (int k = 0; k < NI; ++k) {
          const int c = tx + 16 * k;
          if (c >= r && c < pw) a[i][k] -= ur[i] * uc[k];
        }
      }
    }
    if (j + 1 < pw) {
#pragma unroll
      for (int i = 0; i < NI; ++i)
        if (ty + 16 * i == j + 1)
#pragma unroll
          for (int k = 0; k < NI; ++k) rowbuf[(j + 1) & 1][tx + 16 * k] = a[i][k];
    }
  }
  // U to LDS (column reads below), then X = U^{-1} bottom-up in registers (t = partial sums, then X)
#pragma unroll
  for (int i = 0; i < NI; ++i)
#pragma unroll
    for (int k = 0; k < NI; ++k) sU[ty + 16 * i][tx + 16 * k] = a[i][k];
  __syncthreads();
  T t[NI][NI];
#pragma unroll
  for (int i = 0; i < NI; ++i)
#pragma unroll
    for (int k = 0; k < NI; ++k) t[i][k] = (T)0;
  {
    const int last = pw - 1;
#pragma unroll
    for (int i = 0; i < NI; ++i)
      if (ty + 16 * i == last)
#pragma unroll
        for (int k = 0; k < NI; ++k) {
          const int c = tx + 16 * k;
          const T x = (c == last) ? (T)1 / sU[last][last] : (T)0;
          t[i][k] = x;
          rowbuf[last & 1][c] = x;
        }
  }
  for (int i0 = pw - 1; i0 >= 0; --i0) {
    __syncthreads();
    const T* xb = rowbuf[i0 & 1];
    T xc[NI];
#pragma unroll
    for (int k = 0; k < NI; ++k) xc[k] = xb[tx + 16 * k];
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int r = ty + 16 * i;
      if (r < i0) {
        const T uri = sU[r][i0];
#pragma unroll
        for (int k = 0; k < NI; ++k) t[i][k] += uri * xc[k];
      }
    }
    const int nr = i0 - 1;  // row finalized in this step
    if (nr >= 0) {
      const T inv = (T)1 / sU[nr][nr];
#pragma unroll
      for (int i = 0; i < NI; ++i)
        if (ty + 16 * i == nr)
#pragma unroll
          for (int k = 0; k < NI; ++k) {
            const int c = tx + 16 * k;
            const T x = (c >= nr && c < pw) ? ((c == nr ? (T)1 : (T)0) - t[i][k]) * inv : (T)0;
            t[i][k] = x;
            rowbuf[nr & 1][c] = x;
          }
    }
  }
#pragma unroll
  for (int i = 0; i < NI; ++i)
#pragma unroll
    for (int k = 0; k < NI; ++k) {
      const int r = ty + 16 * i, c = tx + 16 * k;
      if (r < pw && c < pw) F[(p + r) * d + p + c] = (c >= r) ? t[i][k] : (T)0;
    }
}

// ------------------------------------------------------------------ diagonal block, float, blocked by 32

// acc += Aop Bop for one 32 x 32 block with K = 32 from LDS (fp32 MFMA 32x32x2, 16 steps):
// Aop[i][k] = Am[i * lda + k] (a_rows) or Am[k * lda + i]; Bop[k][j] = Bm[k * ldb + j].
LOCA_DEV void mm32(f32x16_t& acc, const float* Am, int lda, bool a_rows, const float* Bm, int ldb, int lane) {
  const int i = lane & 31, kh = lane >> 5;
#pragma unroll
  for (int s2 = 0; s2 < 32; s2 += 2) {
    const int k = s2 + kh;
    const float av = a_rows ? Am[i * lda + k] : Am[k * lda + i];
    acc = mfma_f32x2(av, Bm[k * ldb + i], acc);
  }
}
LOCA_DEV void zero16(f32x16_t& acc) {
#pragma unroll
  for (int r = 0; r < 16; ++r) acc[r] = 0.f;
}

// One wave factors the 32 x 32 block B (upper part used) as U^T U, writes U over B (zero
// below the diagonal) and X = U^{-1} to Xo.  Lane c < 32 holds column c (rows 0..31);
// lanes 32..63 mirror lanes 0..31 and write nothing.  Step j of the factorization takes
// the pivot from lane j (v_readlane; lane j forms it in step j - 1 from its own values,
// so that the pivot does not wait for the row's round trip through LDS) and writes row j of
// U, U[j][c] from lane c, straight to its place in B; the update A[i][c] -= U[j][i] U[j][c]
// then reads that row back from LDS (one broadcast read per entry instead of a cross-lane
// read each).  The inverse is
// built bottom-up the same way, lane c finishing column c of X with row i of U read from
// B.  A wave's LDS accesses complete in order, so each read sees the row just written.
// 1/sqrt of the pivot and the reciprocals are the hardware ones (about 1 ulp).  The first
// non-positive pivot among the first `valid` is reported (1-based, offset base).
LOCA_DEV float lane_val(float v, int l) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}
LOCA_DEV void chol_inv32(float* B, int ld, float* Xo, int ldx, int lane, int valid, int64_t base, int32_t* info) {
  const int c = lane & 31;
  const bool wr = lane < 32;
  float a[32];
#pragma unroll
  for (int r = 0; r < 32; ++r) a[r] = B[r * ld + c];
  float piv = lane_val(a[0], 0);
  int bad = 32;  // the first non-positive pivot (wave-uniform), reported after the loop
#pragma unroll
  for (int j = 0; j < 32; ++j) {
    if (!(piv > 0.f) && j < valid && bad == 32) bad = j;
    const float inv = __builtin_amdgcn_rsqf(piv);
    const float ujj = piv * inv;
    const float uc = c > j ? a[j] * inv : (c == j ? ujj : 0.f);  // U[j][c]
    a[j] = uc;
    // the next pivot from lane j + 1's own values (U[j][j + 1] is its uc), ahead of the
    // row's round trip through LDS; the same fused operation as its update below
    if (j < 31) piv = lane_val(fmaf(-uc, uc, a[j + 1]), j + 1);
    if (wr) B[j * ld + c] = uc;
#pragma unroll
    for (int i = j + 1; i < 32; ++i) a[i] = fmaf(-B[j * ld + i], uc, a[i]);  // A[i][c] -= U[j][i] U[j][c]
  }
  if (bad < 32 && lane == 0) atomicCAS(info, 0, (int32_t)(base + bad + 1));
  float x[32];
#pragma unroll
  for (int i = 31; i >= 0; --i) {
    float part[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int k = i + 1; k < 32; ++k) part[k & 3] += B[i * ld + k] * x[k];  // U[i][k] x[k]
    const float tot = (part[0] + part[1]) + (part[2] + part[3]);
    x[i] = c >= i ? ((c == i ? 1.f : 0.f) - tot) * __builtin_amdgcn_rcpf(B[i * ld + i]) : 0.f;
  }
  if (wr) {
#pragma unroll
    for (int r = 0; r < 32; ++r) Xo[r * ldx + c] = x[r];
  }
}

// Factor and invert the P x P (P = 128) diagonal block of F at p, blocked by 32: per
// 32-column block q, one wave factors and inverts the block (chol_inv32), the waves form
// its row panel U_qr = X_qq^T A_qr and the update A_rs -= U_qr^T U_qs with MFMA; the
// inverse of the whole block is then assembled column by column (wave s):
// X_rs = -X_rr sum_{r < t <= s} U_rt X_ts.  Entries past the matrix (a ragged last block)
// are an identity extension.  Output as for k_diag_block: X over the diagonal block, zero
// strictly below its diagonal.
__global__ __launch_bounds__(kT) void k_diag_f32(int64_t d, int64_t p, float* __restrict__ Fall,
                                                 int32_t* __restrict__ dev_info) {
  constexpr int P = 128, LD = 132;
  __shared__ __attribute__((aligned(16))) float sA[P * LD];
  __shared__ __attribute__((aligned(16))) float sX[P * LD];
  __shared__ __attribute__((aligned(16))) float sT[3][32 * 36];
  const int64_t mi = blockIdx.x;
  float* F = Fall + mi * d * d;
  const float* A0 = F + p * d + p;
  const int pw = (int)((d - p) < P ? (d - p) : P);
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  // the block in 16 four-column chunks per thread, all loads issued before the first use
  // (16-byte loads when the rows are 16-byte aligned and the chunk lies inside the block)
  {
    constexpr int NCH = P * P / 4 / kT;
    float4 v[NCH];
    if ((d & 3) == 0 && pw == P) {  // a whole block with 16-byte aligned rows
#pragma unroll
      for (int u = 0; u < NCH; ++u) {
        const int e = tid + kT * u, r = e >> 5, c = 4 * (e & 31);
        v[u] = *(const float4*)(A0 + (int64_t)r * d + c);
      }
    } else {
#pragma unroll
      for (int u = 0; u < NCH; ++u) {
        const int e = tid + kT * u, r = e >> 5, c = 4 * (e & 31);
        const int64_t o = (int64_t)r * d + c;
        v[u].x = ld_or_zero(A0, o, r < pw && c < pw);
        v[u].y = ld_or_zero(A0, o + 1, r < pw && c + 1 < pw);
        v[u].z = ld_or_zero(A0, o + 2, r < pw && c + 2 < pw);
        v[u].w = ld_or_zero(A0, o + 3, r < pw && c + 3 < pw);
      }
    }
#pragma unroll
    for (int u = 0; u < NCH; ++u) {
      const int e = tid + kT * u, r = e >> 5, c = 4 * (e & 31);
      const float in4[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
      float o4[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int cc = c + t;
        const bool in = r < pw && cc < pw;
        o4[t] = in ? (cc >= r ? in4[t] : 0.f) : (r == cc ? 1.f : 0.f);
      }
      *(float4*)&sA[r * LD + c] = make_float4(o4[0], o4[1], o4[2], o4[3]);
      *(float4*)&sX[r * LD + c] = make_float4(0.f, 0.f, 0.f, 0.f);
    }
  }
  __syncthreads();
  for (int q = 0; q < 4; ++q) {
    const int c0 = 32 * q;
    if (wid == 0) chol_inv32(sA + c0 * LD + c0, LD, sX + c0 * LD + c0, LD, lane, pw - c0, p + c0, dev_info + mi);
    __syncthreads();
    const int nr = 3 - q;
    if (wid < nr) {  // row panel block r: U_qr = X_qq^T A_qr
      const int r = q + 1 + wid;
      f32x16_t acc;
      zero16(acc);
      mm32(acc, sX + c0 * LD + c0, LD, false, sA + c0 * LD + 32 * r, LD, lane);
#pragma unroll
      for (int e = 0; e < 16; ++e) sA[(c0 + mfma32_row(lane, e)) * LD + 32 * r + (lane & 31)] = acc[e];
    }
    __syncthreads();
    for (int u = wid; u < nr * (nr + 1) / 2; u += 4) {  // trailing block (r, s), q < r <= s
      int r = q + 1, rem = u;
      while (rem >= 4 - r) { rem -= 4 - r; ++r; }
      const int s2 = r + rem;
      f32x16_t acc;
      zero16(acc);
      mm32(acc, sA + c0 * LD + 32 * r, LD, false, sA + c0 * LD + 32 * s2, LD, lane);
#pragma unroll
      for (int e = 0; e < 16; ++e) sA[(32 * r + mfma32_row(lane, e)) * LD + 32 * s2 + (lane & 31)] -= acc[e];
    }
    __syncthreads();
  }
  if (wid >= 1) {  // column s = wid of the inverse
    const int s2 = wid;
    float* T = sT[wid - 1];
    for (int r = s2 - 1; r >= 0; --r) {
      f32x16_t acc;
      zero16(acc);
      for (int t = r + 1; t <= s2; ++t) mm32(acc, sA + 32 * r * LD + 32 * t, LD, true, sX + 32 * t * LD + 32 * s2, LD, lane);
#pragma unroll
      for (int e = 0; e < 16; ++e) T[mfma32_row(lane, e) * 36 + (lane & 31)] = acc[e];
      zero16(acc);
      mm32(acc, sX + 32 * r * LD + 32 * r, LD, true, T, 36, lane);
#pragma unroll
      for (int e = 0; e < 16; ++e) sX[(32 * r + mfma32_row(lane, e)) * LD + 32 * s2 + (lane & 31)] = -acc[e];
    }
  }
  __syncthreads();
  for (int e = tid; e < P * P / 4; e += kT) {
    const int r = e >> 5, c = 4 * (e & 31);
    if (r >= pw) continue;
    const float4 x = *(const float4*)&sX[r * LD + c];
    const float x4[4] = {c >= r ? x.x : 0.f, c + 1 >= r ? x.y : 0.f, c + 2 >= r ? x.z : 0.f, c + 3 >= r ? x.w : 0.f};
    float* dst = F + (p + r) * d + p + c;
    if ((d & 3) == 0 && c + 4 <= pw) {
      *(float4*)dst = make_float4(x4[0], x4[1], x4[2], x4[3]);
    } else {
#pragma unroll
      for (int t = 0; t < 4; ++t)
        if (c + t < pw) dst[t] = x4[t];
    }
  }
}

// ------------------------------------------------------------------ panel products (row panel, trailing update)

LOCA_DEV void upper_tile_c(int u, int T, int& I, int& J) {
  int i = 0;
  while (u >= T - i) { u -= T - i; ++i; }
  I = i;
  J = i + u;
}

// Out[i][j] (op)= sum_{kk < K} Pn[kk][i] Qn[kk][j] for one P x P output tile, with the
// K rows streamed through LDS in chunks of kKC rows, double-buffered via registers.
//   kRowPanel: Pn = U11^{-1} (diagonal block), Qn = the chunk's columns of the row
//              panel (F or R), Out = the same chunk, overwritten: U12 = U11^{-T} A12;
//   kTrailing: Pn, Qn = the row panel U12 (F) / its RHS rows (R), Out -= on the upper
//              tiles of the trailing matrix and on the RHS rows below the panel.
constexpr int kKC = 32;
enum PanelJob { kRowPanel = 0, kTrailing = 1 };

// kTrailing takes its K rows from [k0, k0 + kw) of F and R and updates the region of
// rows and columns >= off: every upper tile plus the RHS rows (strip = 0), or only the
// first row of tiles, rows [off, off + P) (strip = 1).  Job = blockIdx.x + job0, the
// upper tiles first, then the RHS tiles.
template <typename T, int JOB>
__global__ __launch_bounds__(kT) __attribute__((amdgpu_waves_per_eu(2))) void k_panel_product(
    int64_t d, int64_t m, int64_t p, int64_t k0, int64_t kw, int64_t off, int strip, int job0, T* __restrict__ Fall,
    T* __restrict__ Rall) {
  constexpr int P = Mf<T>::P, LD = P + 4, PER = (kKC * P) / kT;
  __shared__ T sP[2][kKC * LD];
  __shared__ T sQ[2][kKC * LD];
  const int64_t mi = blockIdx.y;
  T* F = Fall + mi * d * d;
  T* R = Rall + mi * d * m;
  const int pw = JOB == kRowPanel ? (int)((d - p) < P ? (d - p) : P) : (int)kw;  // K rows
  if (JOB == kRowPanel) off = p + pw;
  const int64_t nrem = d - off;
  const int64_t nchF = (nrem + P - 1) / P;
  bool rhs, diag = false;
  int64_t orow, ocol, ocend;  // output tile origin (row in F/R, column) and column end
  const T* gP;                // row kk of Pn at gP + kk * ldp, column i at + i
  const T* gQ;
  int64_t ldq, prows_ok;
  if (JOB == kRowPanel) {
    const int64_t job = (int64_t)blockIdx.x + job0;
    rhs = job >= nchF;
    ocol = rhs ? (job - nchF) * P : off + job * P;
    ocend = rhs ? m : d;
    orow = p;
    gP = F + p * d + p;
    prows_ok = pw;
    gQ = rhs ? R + p * m + ocol : F + p * d + ocol;
    ldq = rhs ? m : d;
  } else {
    const int T2 = (int)((nrem + P - 1) / P);
    const int nU = strip ? T2 : T2 * (T2 + 1) / 2;
    const int TM = (int)((m + P - 1) / P);
    const int job = (int)blockIdx.x + job0;
    int I, J;
    rhs = job >= nU;
    if (!rhs) {
      if (strip) { I = 0; J = job; }
      else upper_tile_c(job, T2, I, J);
    } else { const int u = job - nU; I = u / TM; J = u % TM; }
    diag = !rhs && I == J;
    orow = off + (int64_t)I * P;
    ocol = rhs ? (int64_t)J * P : off + (int64_t)J * P;
    ocend = rhs ? m : d;
    gP = F + k0 * d + orow;
    prows_ok = d - orow;  // columns of Pn that exist
    gQ = rhs ? R + k0 * m + ocol : F + k0 * d + ocol;
    ldq = rhs ? m : d;
  }
  const int64_t pcols_ok = (JOB == kRowPanel) ? pw : prows_ok;
  const int64_t qcols_ok = ocend - ocol;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wid = tid >> 6, wi = wid >> 1, wj = wid & 1;
  const bool active = !(diag && wi > wj);  // strictly lower quarter of a diagonal tile

  T rp[PER], rq[PER];
  auto load_chunk = [&](int kc0) {
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      const int e = tid + q * kT;
      const int kk = e / P, c = e % P;
      const bool okk = kc0 + kk < pw;
      rp[q] = ld_or_zero(gP, (int64_t)(kc0 + kk) * d + c, okk && c < pcols_ok);
      rq[q] = ld_or_zero(gQ, (int64_t)(kc0 + kk) * ldq + c, okk && c < qcols_ok);
    }
  };
  auto store_chunk = [&](int buf) {
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      const int e = tid + q * kT;
      sP[buf][(e / P) * LD + e % P] = rp[q];
      sQ[buf][(e / P) * LD + e % P] = rq[q];
    }
  };

  typename Mf<T>::acc_t acc[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) acc[a][b] = Mf<T>::zero();
  const int nk = (pw + kKC - 1) / kKC;
  load_chunk(0);
  store_chunk(0);
  __syncthreads();
  for (int kc = 0; kc < nk; ++kc) {
    const int cur = kc & 1;
    if (kc + 1 < nk) load_chunk((kc + 1) * kKC);
    if (active) tile_mma<T>(sP[cur], sQ[cur], LD, kKC, wi, wj, lane, acc);
    if (kc + 1 < nk) store_chunk(cur ^ 1);
    __syncthreads();
  }
  if (!active) return;
  T* Out = rhs ? R : F;
  const int64_t ldo = rhs ? m : d;
  const int64_t rend = (JOB == kRowPanel) ? p + pw : d;
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      T old[Mf<T>::NR];
      const int64_t col = ocol + wj * (P / 2) + b * Mf<T>::BLK + Mf<T>::col(lane);
      const int64_t rbase = orow + wi * (P / 2) + a * Mf<T>::BLK;
#pragma unroll
      for (int r = 0; r < Mf<T>::NR; ++r) {
        const int64_t row = rbase + Mf<T>::row(lane, r);
        const bool ok = row < rend && col < ocend && (JOB == kRowPanel || rhs || col >= row);
        if (JOB == kTrailing) old[r] = ld_or_zero(Out, row * ldo + col, ok);
      }
#pragma unroll
      for (int r = 0; r < Mf<T>::NR; ++r) {
        const int64_t row = rbase + Mf<T>::row(lane, r);
        const bool ok = row < rend && col < ocend && (JOB == kRowPanel || rhs || col >= row);
        if (ok) Out[row * ldo + col] = (JOB == kTrailing) ? old[r] - acc[a][b][r] : acc[a][b][r];
      }
    }
}

// ------------------------------------------------------------------ trailing update on bf16 matrix cores

// A float a is carried as three bfloat16 parts, h = bf16(a), m = bf16(a - h),
// l = bf16(a - h - m) (each difference is exact in float), which hold a to about 2^-27
// relative.  The product of two split values keeps the six terms of order 2^-16 and
// larger (h*h, h*m, m*h, h*l, l*h, m*m) and drops m*l, l*m, l*l (order 2^-24 and
// below), so the update has float-class error while running on bf16 MFMA, which
// retires sixteen times the flops of the fp32 MFMA per cycle.
// The split is split3_pair (loca_bf16.h): hardware conversions, two values at a time.

// Panel products on bf16 matrix cores, Out[i][j] (op)= sum_kk Pn[kk][i] Qn[kk][j]:
//   kX6Trail: F[i][j] -= sum_{kk in [k0, k0 + kw)} F[kk][i] F[kk][j] on the upper
//             256 x 256 tiles of the trailing region [off, d);
//   kX6Strip: the same for the rows [off, off + 128) only (128 x 256 tiles, columns
//             from off), the update of a panel by the earlier panels of its super-panel;
//   kX6Row:   F[p + i][j] = sum_kk X[kk][i] F[p + kk][j] for the columns j >= p + 128 of
//             the panel rows (128 x 256 tiles), X = U11^{-1} in the diagonal block.
// A stage is 16 rows of K: each operand is loaded into registers several stages ahead (a
// ring of D stages), split, and written to LDS as three bf16 planes [16][LD]; eight waves
// (2 x 4) read their MFMA operands with transpose reads (LD = 288: the four rows a
// half-wave reads start 64 bytes apart modulo 256, so the reads are conflict-free).
// Requires d % 4 == 0.
constexpr int kX6BK = 16, kX6LD = 288;
enum X6Mode { kX6Trail = 0, kX6Strip = 1, kX6Row = 2, kX6TrailRhs = 3 };

LOCA_DEV float4 ld4_or_zero(const float* base, int64_t idx, bool ok) {
  const float4 v = *(const float4*)(base + (ok ? idx : 0));
  return ok ? v : make_float4(0.f, 0.f, 0.f, 0.f);
}
LOCA_DEV float4 ld4_or_zero_ro(const float* __restrict__ base, int64_t idx, bool ok) { return ld4_or_zero(base, idx, ok); }

// Jobs past the nF tiles of F are right-hand-side jobs: the same product with Qn and the
// output taken from R (d x m per matrix, m % 4 == 0): the 256-row block u of the trailing
// region (kX6Trail), or the panel rows (kX6Strip, kX6Row), all m columns.
// kX6TrailRhs: only the right-hand-side jobs of kX6Trail, in a layout for their few
// columns: a workgroup takes 256 rows x 32 columns (eight waves of 32 x 32; columns
// 32 blockIdx.z ..), so it does an eighth of the matrix-core work of a 256 x 256 tile.
template <int MODE>
__global__ __launch_bounds__(512) void k_panel_x6(int64_t d, int64_t k0, int64_t kw, int64_t off,
                                                  float* __restrict__ Fall, float* __restrict__ Rall, int64_t m,
                                                  int nF) {
  constexpr bool RH = MODE == kX6TrailRhs;
  constexpr int BR = (MODE == kX6Trail || RH) ? 256 : 128;  // output rows per tile
  constexpr int BC = RH ? 32 : 256, WGN = RH ? 1 : 4, WGM = 8 / WGN;
  constexpr int WM = BR / WGM, WN = BC / WGN, NBM = WM / 32, NBN = WN / 32;
  constexpr int LD = kX6LD, PLANE = kX6BK * LD;
  constexpr int NQV = BC * kX6BK / 4;                                  // float4 values of a Qn stage
  constexpr int QP = BR * kX6BK / 4 / 512, QQ = (NQV + 511) / 512;     // float4 loads per thread
  __shared__ __attribute__((aligned(16))) uint16_t sm[2][6 * PLANE];  // [buffer][operand * 3 + part]
  const int64_t mi = blockIdx.y;
  float* F = Fall + mi * d * d;
  float* R = Rall + mi * d * m;
  const bool rhs = RH || (int)blockIdx.x >= nF;
  const int job = rhs && !RH ? (int)blockIdx.x - nF : (int)blockIdx.x;
  int64_t orow, ocol, pcol;
  bool diag = false;
  if (RH) {
    orow = off + (int64_t)job * BR;
    ocol = (int64_t)blockIdx.z * BC;
    pcol = orow;
  } else if (MODE == kX6Trail) {
    if (rhs) {
      orow = off + (int64_t)job * BC;
      ocol = 0;
    } else {
      const int T2 = (int)((d - off + BC - 1) / BC);
      int I, J;
      upper_tile_c(job, T2, I, J);
      diag = I == J;
      orow = off + (int64_t)I * BC;
      ocol = off + (int64_t)J * BC;
    }
    pcol = orow;
  } else if (MODE == kX6Strip) {
    diag = !rhs && job == 0;
    orow = off;
    ocol = rhs ? 0 : off + (int64_t)job * BC;
    pcol = orow;
  } else {  // kX6Row: K rows and output rows [k0, k0 + 128), Pn = the diagonal block
    orow = k0;
    ocol = rhs ? 0 : k0 + 128 + (int64_t)job * BC;
    pcol = k0;
  }
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6, wi = wid / WGN, wj = wid % WGN;
  const bool active = !(diag && (wj + 1) * WN <= wi * WM);
  const float* gP = F + k0 * d + pcol;
  float* Out = rhs ? R : F;                          // Qn and the output
  const int64_t ldq = rhs ? m : d, qend = rhs ? m : d;
  const float* gQ = Out + k0 * ldq + ocol;
  const int64_t pend = MODE == kX6Row ? k0 + 128 : d;  // columns of Pn that exist: < pend

  // a ring of D stages of global loads in flight: the loads of stage kc + D are issued
  // when stage kc is consumed, so D - 1 stages of matrix-core work cover their latency
  constexpr int D = MODE == kX6Trail ? 2 : 4;
  float4 rp[D][QP], rq[D][QQ];
  auto load = [&](int slot, int kc0) {
#pragma unroll
    for (int q = 0; q < QP; ++q) {
      const int c = tid + 512 * q, kk = c / (BR / 4), c4 = 4 * (c % (BR / 4));
      rp[slot][q] = ld4_or_zero(gP, (int64_t)(kc0 + kk) * d + c4, kc0 + kk < kw && pcol + c4 < pend);
    }
#pragma unroll
    for (int q = 0; q < QQ; ++q) {
      const int c = tid + 512 * q, kk = c / (BC / 4), c4 = 4 * (c % (BC / 4));
      if (c < NQV)
        rq[slot][q] = ld4_or_zero(gQ, (int64_t)(kc0 + kk) * ldq + c4, kc0 + kk < kw && ocol + c4 < qend);
    }
  };
  auto put = [&](uint16_t* base, int kk, int c4, const float4& v) {
    uint32_t h[2], m[2], l[2];
    split3_pair(v.x, v.y, h[0], m[0], l[0]);
    split3_pair(v.z, v.w, h[1], m[1], l[1]);
    const int o = kk * LD + c4;
    *(uint2*)(base + o) = make_uint2(h[0], h[1]);
    *(uint2*)(base + PLANE + o) = make_uint2(m[0], m[1]);
    *(uint2*)(base + 2 * PLANE + o) = make_uint2(l[0], l[1]);
  };
  auto store = [&](int buf, int slot) {
#pragma unroll
    for (int q = 0; q < QP; ++q) {
      const int c = tid + 512 * q;
      put(&sm[buf][0], c / (BR / 4), 4 * (c % (BR / 4)), rp[slot][q]);
    }
#pragma unroll
    for (int q = 0; q < QQ; ++q) {
      const int c = tid + 512 * q;
      if (c < NQV) put(&sm[buf][3 * PLANE], c / (BC / 4), 4 * (c % (BC / 4)), rq[slot][q]);
    }
  };

  f32x16_t acc[NBM][NBN];
#pragma unroll
  for (int a = 0; a < NBM; ++a)
#pragma unroll
    for (int b = 0; b < NBN; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.f;

  const int nk = (int)((kw + kX6BK - 1) / kX6BK);
#pragma unroll
  for (int u = 0; u < D; ++u)
    if (u < nk) load(u, u * kX6BK);
  store(0, 0);
  __syncthreads();
  for (int kc0 = 0; kc0 < nk; kc0 += D) {
#pragma unroll
    for (int u = 0; u < D; ++u) {  // stage kc = kc0 + u: in LDS buffer kc & 1; its register slot is u
      const int kc = kc0 + u;
      if (kc >= nk) break;
      const int cur = kc & 1;
      if (kc + D < nk) load(u, (kc + D) * kX6BK);
      bf16x8_t fa[3][NBM], fb[3][NBN];
#pragma unroll
      for (int t = 0; t < 3; ++t) {
#pragma unroll
        for (int a = 0; a < NBM; ++a) fa[t][a] = frag32_tr(&sm[cur][t * PLANE], LD, wi * WM + 32 * a, 0, lane);
#pragma unroll
        for (int b = 0; b < NBN; ++b)
          fb[t][b] = frag32_tr(&sm[cur][(3 + t) * PLANE], LD, wj * WN + 32 * b, 0, lane);
      }
      // the six kept terms, smallest first; each term runs over all blocks, so the MFMAs
      // into one accumulator are NBM * NBN instructions apart
      constexpr int TA[6] = {2, 0, 1, 1, 0, 0}, TB[6] = {0, 2, 1, 0, 1, 0};
#pragma unroll
      for (int t = 0; t < 6; ++t)
#pragma unroll
        for (int a = 0; a < NBM; ++a)
#pragma unroll
          for (int b = 0; b < NBN; ++b) acc[a][b] = mfma32(fa[TA[t]][a], fb[TB[t]][b], acc[a][b]);
      if (kc + 1 < nk) store(cur ^ 1, (u + 1) % D);
      __syncthreads();
    }
  }
  if (!active) return;
  int64_t rend = MODE == kX6Row ? k0 + 128 : (MODE == kX6Strip ? off + 128 : d);
  if (rend > d) rend = d;  // a ragged last panel
#pragma unroll
  for (int a = 0; a < NBM; ++a)
#pragma unroll
    for (int b = 0; b < NBN; ++b) {
      const int64_t col = ocol + wj * WN + 32 * b + mfma32_col(lane);
      const int64_t rb = orow + wi * WM + 32 * a;
      float old[16];
      if (MODE != kX6Row) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int64_t row = rb + mfma32_row(lane, r);
          old[r] = ld_or_zero(Out, row * ldq + col, row < rend && col < qend && (rhs || col >= row));
        }
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t row = rb + mfma32_row(lane, r);
        if (row < rend && col < qend && (rhs || col >= row))
          Out[row * ldq + col] = MODE == kX6Row ? acc[a][b][r] : old[r] - acc[a][b][r];
      }
    }
}

// ------------------------------------------------------------------ trailing update, fp32 rows split in registers

// The trailing update of a super-panel, F[i][j] -= sum_kk U[kk][i] U[kk][j] over its kw rows
// kk in [k0, k0 + kw), on the upper 256 x 256 tiles of the trailing region [off, d), with
// the fp32 rows of U read straight from F.  Stages of 16 rows x 256 columns (16 KB per
// panel) stream into a four-slot LDS ring by direct copies, three stages ahead; the 16-byte
// chunks of stage row r sit XOR-swizzled by 8 (r / 8), so that the two half-waves of an
// operand read (rows r and r + 8) fall on different banks.  The factor of the equilibrated
// matrix (unit diagonal) has |U[kk][i]| <= 1, so every operand, scaled by 2^8, is split in
// registers into two fp16 parts, u = h + l with h = fp16(2^8 u) and l = fp16(2^8 u - h)
// (22 bits of u; a part past the fp16 range cannot occur), and the three kept products
// l h, h l, h h (smallest first) run on the fp16 matrix cores, accumulated in fp32 and
// scaled back by 2^-16 (exact) when F is updated: half the matrix-core work of a three-part
// bf16 split, with product errors of the order of the fp32 accumulation's own rounding.
// A diagonal tile needs one panel (its second ring panel reads nothing).  Tiles, waves and
// the XCD-aware workgroup order are those of the Gram kernel.
// Requires d % 4 == 0, kw % 16 == 0 and 4 d^2 < 2^31 bytes per matrix.
constexpr int kS32BK = 16;  // K rows per stage
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2_v __attribute__((ext_vector_type(2)));
LOCA_DEV f32x16_t mfma32h(f16x8_t a, f16x8_t b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}
// (2^8 a0, 2^8 a1) = h + l as packed fp16 pairs (a0 in the low halves); the difference is
// exact in float
LOCA_DEV void split2h_pair(float a0, float a1, uint32_t& hp, uint32_t& lp) {
  const float s0 = a0 * 256.f, s1 = a1 * 256.f;
  const f32x2_v v = {s0, s1};
  const f16x2_v h = __builtin_convertvector(v, f16x2_v);
  const float r0 = s0 - (float)h[0], r1 = s1 - (float)h[1];
  const f32x2_v r = {r0, r1};
  hp = __builtin_bit_cast(uint32_t, h);
  lp = __builtin_bit_cast(uint32_t, __builtin_convertvector(r, f16x2_v));
}
// the 8 fp32 operand values of lane `lane` (rows 8 (lane / 32) + e of the stage, column
// c0 + lane % 32 of the panel) from a swizzled stage, split into three MFMA operands
LOCA_DEV void frag_f32_split(const float* stage, int c0, int lane, bf16x8_t& fh, bf16x8_t& fm, bf16x8_t& fl) {
  const int hw = lane >> 5, cc = c0 + (lane & 31);
  const float* p = stage + 8 * hw * 256 + 4 * ((cc >> 2) ^ (8 * hw)) + (cc & 3);
  float v[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) v[e] = p[e * 256];
  uint32_t h[4], m[4], l[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) split3_pair(v[2 * e], v[2 * e + 1], h[e], m[e], l[e]);
  fh = __builtin_bit_cast(bf16x8_t, make_uint4(h[0], h[1], h[2], h[3]));
  fm = __builtin_bit_cast(bf16x8_t, make_uint4(m[0], m[1], m[2], m[3]));
  fl = __builtin_bit_cast(bf16x8_t, make_uint4(l[0], l[1], l[2], l[3]));
}
// the 8 fp32 operand values of lane `lane` (as for frag_f32_split), split into two fp16
// MFMA operands of 2^8 times their value
LOCA_DEV void frag_f32_split2h(const float* stage, int c0, int lane, f16x8_t& fh, f16x8_t& fl) {
  const int hw = lane >> 5, cc = c0 + (lane & 31);
  const float* p = stage + 8 * hw * 256 + 4 * ((cc >> 2) ^ (8 * hw)) + (cc & 3);
  float v[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) v[e] = p[e * 256];
  uint32_t h[4], l[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) split2h_pair(v[2 * e], v[2 * e + 1], h[e], l[e]);
  fh = __builtin_bit_cast(f16x8_t, make_uint4(h[0], h[1], h[2], h[3]));
  fl = __builtin_bit_cast(f16x8_t, make_uint4(l[0], l[1], l[2], l[3]));
}
__global__ __launch_bounds__(512) void k_syrk_f32_dl(int64_t d, int64_t k0, int64_t kw, int64_t off,
                                                     float* __restrict__ Fall, int ntile) {
  constexpr int BM = 256, NT = 512, WGN = 4, WM = 128, WN = 64, NBM = WM / 32, NBN = WN / 32;
  constexpr int TILE_F = kS32BK * BM;            // floats of one panel stage
  constexpr int NQ = TILE_F * 4 / 16 / NT;       // 16-byte copies per thread per panel
  constexpr int NCP = 2 * NQ;                    // copies per thread per stage
  static_assert(NCP == NBM, "one copy per fragment row of a stage");
  __shared__ __attribute__((aligned(1024))) float sb0[2 * TILE_F];
  __shared__ __attribute__((aligned(1024))) float sb1[2 * TILE_F];
  __shared__ __attribute__((aligned(1024))) float sb2[2 * TILE_F];
  __shared__ __attribute__((aligned(1024))) float sb3[2 * TILE_F];

  const int T = (int)((d - off + BM - 1) / BM);
  const int logical = xcd_logical((int)blockIdx.x, (int)gridDim.x);
  int I, J;
  upper_tile_c(logical % ntile, T, I, J);
  const int64_t mi = logical / ntile;
  float* F = Fall + mi * d * d;
  const bool diag = I == J;
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int wi = wid / WGN, wj = wid % WGN;
  const bool active = !(diag && (wj + 1) * WN <= wi * WM);
  const int64_t cI = off + (int64_t)I * BM, cJ = off + (int64_t)J * BM;
  const int nk = (int)(kw / kS32BK);

  // copy q of this thread fills LDS chunk position (NQ wid + q) * 64 + lane of a panel stage:
  // stage row slot / 64, position slot % 64, holding global chunk position ^ 8 (row / 8)
  int lrow[NQ], lcol[NQ];
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    const int slot = (NQ * wid + q) * 64 + lane;
    lrow[q] = slot >> 6;
    lcol[q] = 4 * ((slot & 63) ^ (8 * ((slot >> 9) & 1)));
  }
  const i32x4_t rs = buffer_rsrc(F, (uint32_t)(d * d * 4));
  // Copy j of stage kt: panel j / NQ, chunk j % NQ; stages past the last, and the second
  // panel of a diagonal tile, read nothing (out-of-range offsets return zeros).
  auto issue = [&](float* buf, int kt, int j) {
    const int pnl = j / NQ, q = j % NQ;
    const int64_t row = k0 + (int64_t)kt * kS32BK + lrow[q];
    const int64_t col = (pnl == 0 ? cI : cJ) + lcol[q];
    const bool ok = kt < nk && col < d && !(diag && pnl == 1);
    const uint32_t off_b = ok ? (uint32_t)(4 * (row * d + col)) : kBufOutside;
    const uint32_t dst = (uint32_t)(uintptr_t)(LOCA_LDS void*)buf + pnl * TILE_F * 4 + (NQ * wid + q) * 1024;
    lds_dma16_buf(off_b, rs, __builtin_amdgcn_readfirstlane(dst));
  };

  f32x16_t acc[NBM][NBN];
#pragma unroll
  for (int a = 0; a < NBM; ++a)
#pragma unroll
    for (int b = 0; b < NBN; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.f;

  const int bpanel = diag ? 0 : TILE_F;
  auto step = [&](float* cur, float* fill, int kt) {
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(2 * NCP));  // stage kt landed (this thread's copies)
    barrier_nofence();                               // ... everyone's; slot `fill` no longer read
    f16x8_t bh[NBN], bl[NBN];
#pragma unroll
    for (int b = 0; b < NBN; ++b) frag_f32_split2h(cur + bpanel, wj * WN + 32 * b, lane, bh[b], bl[b]);
#pragma unroll
    for (int a = 0; a < NBM; ++a) {
      __builtin_amdgcn_sched_barrier(0);
      issue(fill, kt + 3, a);
      __builtin_amdgcn_sched_barrier(0);
      f16x8_t ah, al;
      frag_f32_split2h(cur, wi * WM + 32 * a, lane, ah, al);
#pragma unroll
      for (int b = 0; b < NBN; ++b) {
        acc[a][b] = mfma32h(al, bh[b], acc[a][b]);
        acc[a][b] = mfma32h(ah, bl[b], acc[a][b]);
        acc[a][b] = mfma32h(ah, bh[b], acc[a][b]);
      }
    }
  };
#pragma unroll
  for (int j = 0; j < NCP; ++j) issue(sb0, 0, j);
#pragma unroll
  for (int j = 0; j < NCP; ++j) issue(sb1, 1, j);
#pragma unroll
  for (int j = 0; j < NCP; ++j) issue(sb2, 2, j);
  for (int kt = 0; kt < nk; kt += 4) {
    step(sb0, sb3, kt);
    if (kt + 1 < nk) step(sb1, sb0, kt + 1);
    if (kt + 2 < nk) step(sb2, sb1, kt + 2);
    if (kt + 3 < nk) step(sb3, sb2, kt + 3);
  }
  __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));  // drain the look-ahead copies before the workgroup ends
  if (!active) return;
#pragma unroll
  for (int a = 0; a < NBM; ++a)
#pragma unroll
    for (int b = 0; b < NBN; ++b) {
      const int64_t col = cJ + wj * WN + 32 * b + mfma32_col(lane);
      const int64_t rb = cI + wi * WM + 32 * a;
      float old[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t row = rb + mfma32_row(lane, r);
        old[r] = ld_or_zero(F, row * d + col, row < d && col < d && col >= row);
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t row = rb + mfma32_row(lane, r);
        if (row < d && col < d && col >= row) F[row * d + col] = old[r] - acc[a][b][r] * (1.0f / 65536.0f);
      }
    }
}

// ------------------------------------------------------------------ back substitution, one row block

// acc[m][q] += sum_kk sA[i][kk] sB[kk][j]: like tile_mma, with the first operand stored
// with K along its rows (row stride lda, odd so that column reads are conflict-free).
template <typename T>
LOCA_DEV void tile_mma_kt(const T* sA, int lda, const T* sB, int ldb, int K, int wi, int wj, int lane,
                          typename Mf<T>::acc_t (&acc)[2][2]) {
  constexpr int BLK = Mf<T>::BLK, KS = Mf<T>::KS, WT = Mf<T>::P / 2;
  const int kr = lane / BLK, cr = lane % BLK;
  for (int kk = 0; kk < K; kk += KS) {
    T a[2], b[2];
#pragma unroll
    for (int m = 0; m < 2; ++m) a[m] = sA[(wi * WT + m * BLK + cr) * lda + kk + kr];
#pragma unroll
    for (int q = 0; q < 2; ++q) b[q] = sB[(kk + kr) * ldb + wj * WT + q * BLK + cr];
#pragma unroll
    for (int m = 0; m < 2; ++m)
#pragma unroll
      for (int q = 0; q < 2; ++q) acc[m][q] = Mf<T>::mma(a[m], b[q], acc[m][q]);
  }
}

// Right-looking back substitution for row block [p, p + pw) of U M' = Y, where the rows
// of R (= Y) have already received the contributions of every block below:
//   M'_p = U11^{-1} R_p                (computed by every workgroup, stored by x == 0)
//   R_r -= U_{r, p:p+pw} M'_p          for the rows r < p of this workgroup's chunk.
// Grid: x = P-row chunks above p (at least one), y = matrix.  The four waves split the
// P rows; each covers NQ MFMA blocks of the m right-hand-side columns (m <= NQ * BLK).
template <typename T, int NQ>
__global__ __launch_bounds__(kT) void k_back_step(int64_t d, int64_t m, int64_t p, const T* __restrict__ Fall,
                                                  T* __restrict__ Rall, T* __restrict__ Mpall) {
  constexpr int P = Mf<T>::P, BLK = Mf<T>::BLK, KS = Mf<T>::KS, NMB = P / 4 / BLK;
  constexpr int NC = NQ * BLK, LDK = P + 1, LDN = NC + 4;
  __shared__ T sA[P * LDK];  // U11^{-1}, then the rows above
  __shared__ T sB[P * LDN];  // R_p, then M'_p
  const int64_t mi = blockIdx.y;
  const T* F = Fall + mi * d * d;
  T* R = Rall + mi * d * m;
  T* Mp = Mpall + mi * d * m;
  const int pw = (int)((d - p) < P ? (d - p) : P);
  const int64_t r0 = (int64_t)blockIdx.x * P;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int kr = lane / BLK, cr = lane % BLK;
  g2s_block<T, P, P, kT>(sA, LDK, F + p * d + p, d, pw, pw);
  g2s_block<T, P, NC, kT>(sB, LDN, R + p * m, m, pw, m);
  __syncthreads();
  typename Mf<T>::acc_t acc[NMB][NQ];
  auto product = [&]() {
#pragma unroll
    for (int x = 0; x < NMB; ++x)
#pragma unroll
      for (int y = 0; y < NQ; ++y) acc[x][y] = Mf<T>::zero();
    for (int kk = 0; kk < pw; kk += KS) {
      T a[NMB], b[NQ];
#pragma unroll
      for (int x = 0; x < NMB; ++x) a[x] = sA[(wid * (P / 4) + x * BLK + cr) * LDK + kk + kr];
#pragma unroll
      for (int y = 0; y < NQ; ++y) b[y] = sB[(kk + kr) * LDN + y * BLK + cr];
#pragma unroll
      for (int x = 0; x < NMB; ++x)
#pragma unroll
        for (int y = 0; y < NQ; ++y) acc[x][y] = Mf<T>::mma(a[x], b[y], acc[x][y]);
    }
  };
  product();
  __syncthreads();  // everyone is done reading sA / sB
#pragma unroll
  for (int x = 0; x < NMB; ++x)
#pragma unroll
    for (int y = 0; y < NQ; ++y)
#pragma unroll
      for (int r = 0; r < Mf<T>::NR; ++r) {
        const int row = wid * (P / 4) + x * BLK + Mf<T>::row(lane, r);
        const int col = y * BLK + Mf<T>::col(lane);
        const T v = (row < pw && col < m) ? acc[x][y][r] : (T)0;
        sB[row * LDN + col] = v;
        if (blockIdx.x == 0 && row < pw && col < m) Mp[(p + row) * m + col] = v;
      }
  if (r0 >= p) return;  // no rows above in this chunk (only chunk 0 exists when p == 0)
  const int64_t rows = (p - r0) < P ? (p - r0) : P;
  g2s_block<T, P, P, kT>(sA, LDK, F + r0 * d + p, d, rows, pw);
  __syncthreads();
  product();
#pragma unroll
  for (int x = 0; x < NMB; ++x)
#pragma unroll
    for (int y = 0; y < NQ; ++y) {
      T old[Mf<T>::NR];
      const int col = y * BLK + Mf<T>::col(lane);
#pragma unroll
      for (int r = 0; r < Mf<T>::NR; ++r) {
        const int row = wid * (P / 4) + x * BLK + Mf<T>::row(lane, r);
        old[r] = ld_or_zero(R, (r0 + row) * m + col, row < rows && col < m);
      }
#pragma unroll
      for (int r = 0; r < Mf<T>::NR; ++r) {
        const int row = wid * (P / 4) + x * BLK + Mf<T>::row(lane, r);
        if (row < rows && col < m) R[(r0 + row) * m + col] = old[r] - acc[x][y][r];
      }
    }
}

// ------------------------------------------------------------------ back substitution, float

// One launch per row block p (descending) of U M' = Y, right-looking, with M'_p already
// in Mp: workgroups x >= 1 apply R_r -= U_{r,p} M'_p to kBackPer row blocks r above p each;
// workgroup 0 applies it to the block q just above p and then forms M'_q = U_qq^{-1} R_q
// (U_qq^{-1} sits in the diagonal block of F), so the next launch finds M'_q in Mp.  With
// `init`, workgroup 0 only forms M'_p of the last block.  The first operand of every
// product streams from F into registers: MFMA j of a K range of 32 takes k = 16 h + j
// in lane half h, for both operands, so a lane reads 16 consecutive floats of its row.
// The second operand (M'_p, or the updated R_q) sits transposed in LDS.
constexpr int kBackPer = 2;  // row blocks per updating workgroup (the launch waits on its slowest)
template <int NQ, bool V4>
__global__ __launch_bounds__(kT) void k_back_f32(int64_t d, int64_t m, int64_t p, int init, const float* __restrict__ Fall,
                                                 float* __restrict__ Rall, float* __restrict__ Mpall) {
  constexpr int P = 128, LDT = P + 4;
  __shared__ __attribute__((aligned(16))) float sT[NQ * 32 * LDT];  // [column][k]
  const int64_t mi = blockIdx.y;
  const float* F = Fall + mi * d * d;
  float* R = Rall + mi * d * m;
  float* Mp = Mpall + mi * d * m;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6, li = lane & 31, h = lane >> 5;
  const int pw = (int)((d - p) < P ? (d - p) : P);

  // acc[q] = sum_{k < kmax} A[32 wid + li][k] T[k][32 q + li] for the wave's 32 rows
  // (rows >= rows_ok of A read as zero)
  auto product = [&](const float* A, int kmax, int rows_ok, f32x16_t (&acc)[NQ]) {
#pragma unroll
    for (int q = 0; q < NQ; ++q)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[q][r] = 0.f;
    const bool rok = 32 * wid + li < rows_ok;
    const float* arow = A + (int64_t)(rok ? 32 * wid + li : 0) * d;
    // the lane's whole row slice (kmax <= P) is loaded before the first product
    float a[P / 2];
#pragma unroll
    for (int kc = 0; kc < P / 32; ++kc) {
      const int kb = 32 * kc + 16 * h;
      if (V4) {
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const float4 t = ld4_or_zero_ro(arow, kb + 4 * v, rok && kb + 4 * v < kmax);
          a[16 * kc + 4 * v] = t.x; a[16 * kc + 4 * v + 1] = t.y; a[16 * kc + 4 * v + 2] = t.z;
          a[16 * kc + 4 * v + 3] = t.w;
        }
      } else {
#pragma unroll
        for (int j = 0; j < 16; ++j) a[16 * kc + j] = ld_or_zero(arow, kb + j, rok && kb + j < kmax);
      }
    }
#pragma unroll
    for (int kc = 0; kc < P / 32; ++kc) {
      if (32 * kc >= kmax) break;
      const int kb = 32 * kc + 16 * h;
#pragma unroll
      for (int q = 0; q < NQ; ++q) {
        const float* tb = sT + (32 * q + li) * LDT + kb;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const float4 t = *(const float4*)(tb + 4 * v);
          acc[q] = mfma_f32x2(a[16 * kc + 4 * v], t.x, acc[q]);
          acc[q] = mfma_f32x2(a[16 * kc + 4 * v + 1], t.y, acc[q]);
          acc[q] = mfma_f32x2(a[16 * kc + 4 * v + 2], t.z, acc[q]);
          acc[q] = mfma_f32x2(a[16 * kc + 4 * v + 3], t.w, acc[q]);
        }
      }
    }
  };
  // sT[c][k] = src[k][c] for k < rows, c < m (zero elsewhere); all loads issued first
  auto load_t = [&](const float* src, int rows) {
    constexpr int PER = NQ * 32 * P / kT;
    float v[PER];
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int e = tid + kT * u, k = e / (NQ * 32), c = e % (NQ * 32);
      v[u] = ld_or_zero(src, (int64_t)k * m + c, k < rows && c < m);
    }
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int e = tid + kT * u, k = e / (NQ * 32), c = e % (NQ * 32);
      sT[c * LDT + k] = v[u];
    }
  };
  auto store_mp = [&](int64_t r0, int rows, const f32x16_t (&acc)[NQ]) {
#pragma unroll
    for (int q = 0; q < NQ; ++q)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = 32 * wid + mfma32_row(lane, r), col = 32 * q + li;
        if (row < rows && col < m) Mp[(r0 + row) * m + col] = acc[q][r];
      }
  };

  f32x16_t acc[NQ];
  if (init) {  // M'_p of the last block from its forward-substituted rows
    load_t(R + p * m, pw);
    __syncthreads();
    product(F + p * d + p, pw, pw, acc);
    store_mp(p, pw, acc);
    return;
  }
  load_t(Mp + p * m, pw);
  __syncthreads();
  const int64_t nab = p / P;  // row blocks above p
  if (blockIdx.x == 0) {
    const int64_t r0 = p - P;
    float rv[NQ][16];
#pragma unroll
    for (int q = 0; q < NQ; ++q)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = 32 * wid + mfma32_row(lane, r), col = 32 * q + li;
        rv[q][r] = ld_or_zero(R, (r0 + row) * m + col, col < m);
      }
    product(F + r0 * d + p, pw, P, acc);
    __syncthreads();  // done with M'_p in LDS
#pragma unroll
    for (int q = 0; q < NQ; ++q)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = 32 * wid + mfma32_row(lane, r), col = 32 * q + li;
        sT[col * LDT + row] = col < m ? rv[q][r] - acc[q][r] : 0.f;
      }
    __syncthreads();
    product(F + r0 * d + r0, P, P, acc);
    store_mp(r0, P, acc);
    return;
  }
  for (int c = 0; c < kBackPer; ++c) {
    const int64_t q0 = nab - 2 - kBackPer * ((int64_t)blockIdx.x - 1) - c;
    if (q0 < 0) break;
    const int64_t r0 = q0 * P;
    // the old values of the block's right-hand sides are loaded before the product
    float old[NQ][16];
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const int col = 32 * q + li;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = 32 * wid + mfma32_row(lane, r);
        old[q][r] = ld_or_zero(R, (r0 + row) * m + col, col < m);
      }
    }
    product(F + r0 * d + p, pw, P, acc);
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const int col = 32 * q + li;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = 32 * wid + mfma32_row(lane, r);
        if (col < m) R[(r0 + row) * m + col] = old[q][r] - acc[q][r];
      }
    }
  }
}

// M = D M' (undo the equilibration), float output.
template <typename T>
__global__ void k_unscale(int64_t d, int64_t m, const T* __restrict__ Rall, const T* __restrict__ Dall,
                          float* __restrict__ Mout, int64_t m_bstride) {
  const int64_t mi = blockIdx.y;
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= d * m) return;
  Mout[mi * m_bstride + e] = (float)(Dall[mi * d + e / m] * Rall[mi * d * m + e]);
}


template <typename T>
size_t solve_ws_t(int64_t nb, int64_t d, int64_t m, int64_t nl, int64_t r_prev) {
  const int64_t nm = nb * nl;
  size_t s = align256(sizeof(T) * nm * d * d);  // F
  s += align256(sizeof(T) * nm * d * m);         // R
  s += align256(sizeof(T) * nm * d);             // D
  s += align256(sizeof(T) * nm * d * m);         // M' (back substitution output)
  s += align256(sizeof(double) * nb * d * (r_prev > 0 ? r_prev : 1));  // S Lp
  s += 256;                                                            // lambdas
  return s;
}

// The launches of a solve group in submission order.  With `ops` null each launch is
// issued at once; otherwise it is kept as a closure (every value it needs copied in) for
// the caller, which interleaves the groups on the host: a group's launches then reach
// its stream while the other groups are still being submitted, instead of after them.
struct Emit {
  std::vector<std::function<hipError_t()>>* ops = nullptr;
  int stagger_at = -1;  // index of the op that records the stagger event, when kept
  hipError_t operator()(std::function<hipError_t()> f) {
    if (!ops) return f();
    ops->push_back(std::move(f));
    return hipSuccess;
  }
};

// The solve of the blocks [b0, b0 + nbg) (all their lambdas) on stream st; workspace
// regions are those of the whole call.  `after_diag`, when given, is recorded after the
// first diagonal-block launch.
template <typename T, typename ST>
hipError_t run_group(const SolveArgs& a, int64_t b0, int64_t nbg, hipStream_t st, T* Fw, T* Rw, T* Dw, T* Mpw,
                     double* SLpw, const double* dlam, hipEvent_t after_diag, Emit& emit) {
  const int64_t d = a.d, m = a.r_prev + a.k, nl = a.n_lambda, nm = nbg * nl, mi0 = b0 * nl;
  T* F = Fw + mi0 * d * d;
  T* R = Rw + mi0 * d * m;
  T* D = Dw + mi0 * d;
  T* Mp = Mpw + mi0 * d * m;
  // trailing updates through the direct-to-LDS kernel when a matrix fits 31-bit byte offsets
  const bool syrk_dl = sizeof(T) == 4 && d % 4 == 0 && 4 * d * d < ((int64_t)1 << 31);
  // an earlier call's factor (fp64 only): only the right-hand-side tiles of each launch run
  const bool reuse = a.reuse_factor && sizeof(T) == 8;
  if (a.reuse_factor && !reuse) return hipErrorNotSupported;
  double* SLp = SLpw + b0 * d * (a.r_prev > 0 ? a.r_prev : 1);
  int32_t* info = a.dev_info + mi0;
  const ST* S = (const ST*)a.S + b0 * a.s_bstride;
  const ST* K = (const ST*)a.K + b0 * a.k_bstride;
  const int64_t r_prev = a.r_prev, s_bstride = a.s_bstride, k_bstride = a.k_bstride;
  const float* lp = a.lp ? a.lp + b0 * a.lp_bstride : nullptr;
  const int64_t lp_bstride = a.lp_bstride;
  hipError_t e = emit([=]() {
    if (r_prev > 0) {
      if (r_prev <= 16) {
        dim3 g((unsigned)((d + kSM - 1) / kSM), (unsigned)nbg, 1);
        k_sym_mul<ST, 16><<<g, 256, 0, st>>>(d, r_prev, S, s_bstride, lp, lp_bstride, SLp);
      } else {
        dim3 g((unsigned)((d + kSM - 1) / kSM), (unsigned)nbg, (unsigned)((r_prev + 31) / 32));
        k_sym_mul<ST, 32><<<g, 256, 0, st>>>(d, r_prev, S, s_bstride, lp, lp_bstride, SLp);
      }
    }
    if (reuse) {  // D and F from the earlier call: the right-hand sides only
      dim3 gr((unsigned)((d * m + 255) / 256), (unsigned)nm);
      k_equil_rhs<T, ST><<<gr, 256, 0, st>>>(d, m, r_prev, K, k_bstride, SLp, (int)nl, D, R);
      return hipGetLastError();
    }
    dim3 g((unsigned)((d + 255) / 256), (unsigned)nm);
    k_equil_diag<T, ST><<<g, 256, 0, st>>>(d, S, s_bstride, dlam, (int)nl, D);
    dim3 g2((unsigned)((d + kEqRows - 1) / kEqRows), (unsigned)nbg);
    bool v4 = false;
    if constexpr (sizeof(T) == 4 && sizeof(ST) == 4)
      v4 = d % 4 == 0 && s_bstride % 4 == 0 && ((uintptr_t)S & 15) == 0;
    if (v4) {
      const dim3 g4((unsigned)((d + kEqRows - 1) / kEqRows), (unsigned)((d + kEqCols - 1) / kEqCols), (unsigned)nbg);
      k_equil_setup_v4<<<g4, kEqCols / 4, 0, st>>>(d, m, r_prev, (const float*)S, s_bstride, (const float*)K,
                                                   k_bstride, SLp, dlam, (int)nl, (const float*)D, (float*)F,
                                                   (float*)R);
    } else {
      k_equil_setup<T, ST><<<g2, 256, 0, st>>>(d, m, r_prev, S, s_bstride, K, k_bstride, SLp, dlam, (int)nl, D, F, R);
    }
    return hipGetLastError();
  });
  if (e != hipSuccess) return e;
  // Blocked right-looking factorization with the forward substitution of the RHS
  // carried along.  The trailing matrix is updated once per super-panel of kSuper
  // panels (one pass over it per kSuper * P columns); inside a super-panel each panel
  // first receives the contributions of the super-panel's earlier panels (a strip
  // update of its own rows), then is factored (diagonal block) and solved (row panel).
  constexpr int P = Mf<T>::P, kSuper = 4;
  const bool x6 = sizeof(T) == 4 && d % 4 == 0;
  const bool x6r = x6 && m % 4 == 0 && m <= 256;  // right-hand sides inside the same launches
  const int64_t TM = (m + P - 1) / P;
  for (int64_t P0 = 0; P0 < d; P0 += kSuper * P) {
    const int64_t P1 = (d - P0) < kSuper * P ? d : P0 + kSuper * P;
    for (int64_t pp = P0; pp < P1; pp += P) {
      const int64_t pw = (d - pp) < P ? (d - pp) : P;
      const int64_t nrem = d - pp - pw;
      const int64_t nchF = (nrem + P - 1) / P;
      if (pp > P0) {
        e = emit([=]() {
          const int64_t T2 = (d - pp + P - 1) / P;
          if (x6) {
            const int nF = (int)((d - pp + 255) / 256);
            k_panel_x6<kX6Strip><<<dim3((unsigned)(nF + (x6r ? 1 : 0)), (unsigned)nm), 512, 0, st>>>(
                d, P0, pp - P0, pp, (float*)F, (float*)R, m, nF);
            if (!x6r)
              k_panel_product<T, kTrailing><<<dim3((unsigned)TM, (unsigned)nm), kT, 0, st>>>(
                  d, m, 0, P0, pp - P0, pp, 1, (int)T2, F, R);
          } else if (reuse) {
            k_panel_product<T, kTrailing><<<dim3((unsigned)TM, (unsigned)nm), kT, 0, st>>>(
                d, m, 0, P0, pp - P0, pp, 1, (int)T2, F, R);
          } else {
            k_panel_product<T, kTrailing><<<dim3((unsigned)(T2 + TM), (unsigned)nm), kT, 0, st>>>(
                d, m, 0, P0, pp - P0, pp, 1, 0, F, R);
          }
          return hipGetLastError();
        });
        if (e != hipSuccess) return e;
      }
      const bool rec = after_diag && pp == 0;
      if (rec && emit.ops) emit.stagger_at = (int)emit.ops->size();
      e = emit([=]() {
        if constexpr (sizeof(T) == 4) k_diag_f32<<<(unsigned)nm, kT, 0, st>>>(d, pp, (float*)F, info);
        else if (!reuse) k_diag_block<T><<<(unsigned)nm, kT, 0, st>>>(d, pp, F, info);
        const hipError_t er = hipGetLastError();
        if (er != hipSuccess || !rec) return er;
        return hipEventRecord(after_diag, st);
      });
      if (e != hipSuccess) return e;
      e = emit([=]() {
        if (x6 && nrem > 0) {
          const int nF = (int)((nrem + 255) / 256);
          k_panel_x6<kX6Row><<<dim3((unsigned)(nF + (x6r ? 1 : 0)), (unsigned)nm), 512, 0, st>>>(
              d, pp, pw, 0, (float*)F, (float*)R, m, nF);
          if (!x6r)
            k_panel_product<T, kRowPanel><<<dim3((unsigned)TM, (unsigned)nm), kT, 0, st>>>(d, m, pp, 0, 0, 0, 0,
                                                                                                 (int)nchF, F, R);
        } else if (reuse) {
          k_panel_product<T, kRowPanel><<<dim3((unsigned)TM, (unsigned)nm), kT, 0, st>>>(d, m, pp, 0, 0, 0, 0,
                                                                                          (int)nchF, F, R);
        } else {
          k_panel_product<T, kRowPanel><<<dim3((unsigned)(nchF + TM), (unsigned)nm), kT, 0, st>>>(
              d, m, pp, 0, 0, 0, 0, 0, F, R);
        }
        return hipGetLastError();
      });
      if (e != hipSuccess) return e;
    }
    if (P1 < d) {
      e = emit([=]() {
        const int64_t T2 = (d - P1 + P - 1) / P, nU = T2 * (T2 + 1) / 2;
        if (x6) {
          const int64_t T6 = (d - P1 + 255) / 256;
          const int nF = (int)(T6 * (T6 + 1) / 2);
          if (syrk_dl) {
            k_syrk_f32_dl<<<dim3((unsigned)(nF * nm)), 512, 0, st>>>(d, P0, P1 - P0, P1, (float*)F, nF);
            if (x6r)
              k_panel_x6<kX6TrailRhs><<<dim3((unsigned)T6, (unsigned)nm, (unsigned)((m + 31) / 32)), 512, 0, st>>>(
                  d, P0, P1 - P0, P1, (float*)F, (float*)R, m, 0);
          } else {
            k_panel_x6<kX6Trail><<<dim3((unsigned)(nF + (x6r ? T6 : 0)), (unsigned)nm), 512, 0, st>>>(
                d, P0, P1 - P0, P1, (float*)F, (float*)R, m, nF);
          }
          if (!x6r)
            k_panel_product<T, kTrailing><<<dim3((unsigned)(T2 * TM), (unsigned)nm), kT, 0, st>>>(
                d, m, 0, P0, P1 - P0, P1, 0, (int)nU, F, R);
        } else if (reuse) {
          k_panel_product<T, kTrailing><<<dim3((unsigned)(T2 * TM), (unsigned)nm), kT, 0, st>>>(
              d, m, 0, P0, P1 - P0, P1, 0, (int)nU, F, R);
        } else {
          k_panel_product<T, kTrailing><<<dim3((unsigned)(nU + T2 * TM), (unsigned)nm), kT, 0, st>>>(
              d, m, 0, P0, P1 - P0, P1, 0, 0, F, R);
        }
        return hipGetLastError();
      });
      if (e != hipSuccess) return e;
    }
  }
  if constexpr (sizeof(T) == 4) {
    const int64_t plast = ((d - 1) / P) * P;
    const int nq = (int)((m + 31) / 32);  // m <= 128 (checked by the API)
    auto back = [=](int64_t pp, int init, unsigned gx) {
      const dim3 grid(gx, (unsigned)nm);
      const bool v4 = d % 4 == 0 && m <= 128;
#define LOCA_BACK(NQ)                                                                                \
  if (v4) k_back_f32<NQ, true><<<grid, kT, 0, st>>>(d, m, pp, init, (const float*)F, (float*)R, (float*)Mp); \
  else k_back_f32<NQ, false><<<grid, kT, 0, st>>>(d, m, pp, init, (const float*)F, (float*)R, (float*)Mp);
      if (nq <= 1) { LOCA_BACK(1) }
      else if (nq <= 2) { LOCA_BACK(2) }
      else { LOCA_BACK(4) }
#undef LOCA_BACK
      return hipGetLastError();
    };
    if ((e = emit([=]() { return back(plast, 1, 1); })) != hipSuccess) return e;
    for (int64_t pp = plast; pp >= P; pp -= P) {
      const int64_t nab = pp / P;
      if ((e = emit([=]() { return back(pp, 0, (unsigned)(1 + (nab - 1 + kBackPer - 1) / kBackPer)); })) != hipSuccess)
        return e;
    }
  } else {
    for (int64_t pp = ((d - 1) / P) * P; pp >= 0; pp -= P) {
      e = emit([=]() {
        const dim3 grid((unsigned)(pp > 0 ? (pp + P - 1) / P : 1), (unsigned)nm);
        const int nq = (int)((m + Mf<T>::BLK - 1) / Mf<T>::BLK);  // m <= 128 (checked by the API)
        if (nq <= 1) k_back_step<T, 1><<<grid, kT, 0, st>>>(d, m, pp, F, R, Mp);
        else if (nq <= 2) k_back_step<T, 2><<<grid, kT, 0, st>>>(d, m, pp, F, R, Mp);
        else if (nq <= 4) k_back_step<T, 4><<<grid, kT, 0, st>>>(d, m, pp, F, R, Mp);
        else k_back_step<T, 8><<<grid, kT, 0, st>>>(d, m, pp, F, R, Mp);
        return hipGetLastError();
      });
      if (e != hipSuccess) return e;
    }
  }
  float* m_out = a.m_out + mi0 * a.m_bstride;
  const int64_t m_bstride = a.m_bstride;
  const bool dense = a.w_dense_out != nullptr;
  if (dense && r_prev != 0) return hipErrorNotSupported;
  const float* cb = dense ? a.credit_b + b0 * a.b_bstride : nullptr;
  const int64_t b_bstride = a.b_bstride, w_bstride = a.w_bstride;
  float* w_out = dense ? a.w_dense_out + mi0 * a.w_bstride : nullptr;
  return emit([=]() {
    k_unscale<T><<<dim3((unsigned)((d * m + 255) / 256), (unsigned)nm), 256, 0, st>>>(d, m, Mp, D, m_out, m_bstride);
    const hipError_t er = hipGetLastError();
    if (er != hipSuccess || !dense) return er;
    // W = M B~ (no earlier adapter: the right factor is B~ alone)
    return launch_lowrank_product(st, nm, d, d, m, m_out, m_bstride, m, cb, b_bstride, nl, d, w_out, w_bstride);
  });
}

// Extra streams and events per device, made on first use: the only state the library
// keeps.  The blocks of a call are split into up to kGroups groups on the caller's stream
// and kGroups - 1 internal streams, group g started once group g - 1 has factored its
// first diagonal block: the latency-bound launches of one group (diagonal blocks, strips,
// back substitution: few workgroups each) then run beside the matrix-core updates of the
// others instead of leaving most of the GPU idle.
//
// The streams and events are shared by every call on a device, so creating them and the
// whole submission of a call that uses them (fork record, waits, launches, join records)
// happen under the device's mutex.  A wait on an event takes the event's state at the time
// the wait is enqueued, so once a call has left the critical section its internal work is
// ordered behind its own fork point and the next call may record the events again.
#ifndef LOCA_SOLVE_GROUPS
#define LOCA_SOLVE_GROUPS 3
#endif
constexpr int kGroups = LOCA_SOLVE_GROUPS;
constexpr int kMaxDevices = 64;
struct Aux {
  std::mutex mu;
  bool ready = false;
  hipStream_t s[kGroups] = {};
  hipEvent_t fork = nullptr;
  hipEvent_t stagger[kGroups] = {};
  hipEvent_t join[kGroups] = {};
};
Aux g_aux[kMaxDevices];

// With the device's mutex held: the internal streams and events exist.
hipError_t aux_ready(Aux& x) {
  if (x.ready) return hipSuccess;
  hipError_t e;
  for (int g = 1; g < kGroups; ++g) {
    if (!x.stagger[g] && (e = hipEventCreateWithFlags(&x.stagger[g], hipEventDisableTiming)) != hipSuccess) return e;
    if (!x.join[g] && (e = hipEventCreateWithFlags(&x.join[g], hipEventDisableTiming)) != hipSuccess) return e;
    if (!x.s[g] && (e = hipStreamCreateWithFlags(&x.s[g], hipStreamNonBlocking)) != hipSuccess) return e;
  }
  if (!x.fork && (e = hipEventCreateWithFlags(&x.fork, hipEventDisableTiming)) != hipSuccess) return e;
  x.ready = true;
  return hipSuccess;
}

template <typename T, typename ST>
hipError_t run_solve(const SolveArgs& a) {
  const int64_t d = a.d, m = a.r_prev + a.k, nl = a.n_lambda, nm = a.nb * nl;
  char* p = a.ws;
  T* F = (T*)p; p += align256(sizeof(T) * nm * d * d);
  T* R = (T*)p; p += align256(sizeof(T) * nm * d * m);
  T* D = (T*)p; p += align256(sizeof(T) * nm * d);
  T* Mp = (T*)p; p += align256(sizeof(T) * nm * d * m);
  double* SLp = (double*)p;
  Lams lams;
  for (int i = 0; i < 8; ++i) lams.v[i] = (i < nl) ? a.lambdas[i] : 0.0;
  double* dlam = (double*)(p + align256(sizeof(double) * a.nb * d * (a.r_prev > 0 ? a.r_prev : 1)));
  // the host lambdas travel by value into a one-wave kernel (no copy from pageable memory)
  k_set_lambdas<<<1, 64, 0, a.stream>>>(lams, dlam, (int)nl);
  k_fill_zero_i32<<<(unsigned)((nm + 255) / 256), 256, 0, a.stream>>>(a.dev_info, nm);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int G = (int)(a.nb < kGroups ? a.nb : kGroups);
  if (G < 2) {
    Emit now;
    return run_group<T, ST>(a, 0, a.nb, a.stream, F, R, D, Mp, SLp, dlam, nullptr, now);
  }
  int dev = 0;
  if ((e = hipGetDevice(&dev)) != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  Aux* x = &g_aux[dev];
  std::lock_guard<std::mutex> hold(x->mu);
  if ((e = aux_ready(*x)) != hipSuccess) return e;
  if ((e = hipEventRecord(x->fork, a.stream)) != hipSuccess) return e;
  // Every group's launches are recorded first, then submitted round-robin, one launch
  // per group in turn.  Group g joins once group g - 1 has submitted its first diagonal
  // block and the event after it; its stream waits for that event, so its GPU work
  // starts behind that block.
  std::vector<std::function<hipError_t()>> ops[kGroups];
  int stagger_at[kGroups];
  hipStream_t sts[kGroups];
  for (int g = 0; g < G; ++g) {
    const int64_t b0 = a.nb * g / G, b1 = a.nb * (g + 1) / G;
    sts[g] = g == 0 ? a.stream : x->s[g];
    hipEvent_t after = g + 1 < G ? x->stagger[g + 1] : nullptr;
    Emit keep;
    keep.ops = &ops[g];
    if ((e = run_group<T, ST>(a, b0, b1 - b0, sts[g], F, R, D, Mp, SLp, dlam, after, keep)) != hipSuccess) return e;
    stagger_at[g] = keep.stagger_at;
    if (after && keep.stagger_at < 0) return hipErrorUnknown;  // every group has a first diagonal block
  }
  size_t pos[kGroups] = {};
  bool joined[kGroups] = {};
  joined[0] = true;
  for (bool left = true; left;) {
    left = false;
    for (int g = 0; g < G; ++g) {
      if (!joined[g]) {
        if (!joined[g - 1] || pos[g - 1] <= (size_t)stagger_at[g - 1]) {
          left = true;
          continue;
        }
        if ((e = hipStreamWaitEvent(sts[g], x->fork, 0)) != hipSuccess) return e;
        if ((e = hipStreamWaitEvent(sts[g], x->stagger[g], 0)) != hipSuccess) return e;
        joined[g] = true;
      }
      if (pos[g] < ops[g].size()) {
        if ((e = ops[g][pos[g]++]()) != hipSuccess) return e;
        left = left || pos[g] < ops[g].size();
      }
    }
  }
  for (int g = 1; g < G; ++g) {
    if ((e = hipEventRecord(x->join[g], x->s[g])) != hipSuccess) return e;
    if ((e = hipStreamWaitEvent(a.stream, x->join[g], 0)) != hipSuccess) return e;
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
