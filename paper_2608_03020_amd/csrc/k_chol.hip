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
#include "loca_common.h"

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
    rhs = (int64_t)blockIdx.x >= nchF;
    ocol = rhs ? ((int64_t)blockIdx.x - nchF) * P : off + (int64_t)blockIdx.x * P;
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
LOCA_DEV void split3(float a, uint16_t& h, uint16_t& m, uint16_t& l) {
  h = f32_to_bf16(a);
  const float r1 = a - bf16_to_f32(h);
  m = f32_to_bf16(r1);
  l = f32_to_bf16(r1 - bf16_to_f32(m));
}

// F[i][j] -= sum_{kk in [k0, k0 + kw)} F[kk][i] F[kk][j] on the upper 256 x 256 tiles of
// the trailing region [off, d) (grid: x = tile, y = matrix).  A stage is 16 rows of K:
// each operand (32 KB of float) is loaded into registers one stage ahead, split, and
// written to LDS as three bf16 planes [16][LD]; eight waves of 128 x 64 read their
// MFMA operands with transpose reads (LD = 288: the four rows a half-wave reads start
// 64 bytes apart modulo 256, so the reads are conflict-free).  Requires d % 4 == 0.
constexpr int kX6BK = 16, kX6LD = 288;

LOCA_DEV float4 ld4_or_zero(const float* base, int64_t idx, bool ok) {
  const float4 v = *(const float4*)(base + (ok ? idx : 0));
  return ok ? v : make_float4(0.f, 0.f, 0.f, 0.f);
}

__global__ __launch_bounds__(512) void k_trail_x6(int64_t d, int64_t k0, int64_t kw, int64_t off,
                                                  float* __restrict__ Fall) {
  constexpr int BM = 256, WGN = 4, WM = 128, WN = 64, NBM = WM / 32, NBN = WN / 32;
  constexpr int LD = kX6LD, PLANE = kX6BK * LD;
  __shared__ __attribute__((aligned(16))) uint16_t sm[2][6 * PLANE];  // [buffer][operand * 3 + part]
  const int64_t mi = blockIdx.y;
  float* F = Fall + mi * d * d;
  const int T2 = (int)((d - off + BM - 1) / BM);
  int I, J;
  upper_tile_c((int)blockIdx.x, T2, I, J);
  const bool diag = I == J;
  const int64_t orow = off + (int64_t)I * BM, ocol = off + (int64_t)J * BM;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6, wi = wid / WGN, wj = wid % WGN;
  const bool active = !(diag && (wj + 1) * WN <= wi * WM);
  const float* gP = F + k0 * d + orow;
  const float* gQ = F + k0 * d + ocol;

  // staging: float4 chunk c = tid + 512 q of the 16 x 64 chunks of an operand stage
  float4 rp[2], rq[2];
  auto load = [&](int kc0) {
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int c = tid + 512 * q, kk = c >> 6, c4 = 4 * (c & 63);
      const bool okk = kc0 + kk < kw;
      rp[q] = ld4_or_zero(gP, (int64_t)(kc0 + kk) * d + c4, okk && orow + c4 < d);
      rq[q] = ld4_or_zero(gQ, (int64_t)(kc0 + kk) * d + c4, okk && ocol + c4 < d);
    }
  };
  auto put = [&](uint16_t* base, int kk, int c4, const float4& v) {
    uint16_t h[4], m[4], l[4];
    split3(v.x, h[0], m[0], l[0]);
    split3(v.y, h[1], m[1], l[1]);
    split3(v.z, h[2], m[2], l[2]);
    split3(v.w, h[3], m[3], l[3]);
    const int o = kk * LD + c4;
    *(uint2*)(base + o) = make_uint2(h[0] | ((uint32_t)h[1] << 16), h[2] | ((uint32_t)h[3] << 16));
    *(uint2*)(base + PLANE + o) = make_uint2(m[0] | ((uint32_t)m[1] << 16), m[2] | ((uint32_t)m[3] << 16));
    *(uint2*)(base + 2 * PLANE + o) = make_uint2(l[0] | ((uint32_t)l[1] << 16), l[2] | ((uint32_t)l[3] << 16));
  };
  auto store = [&](int buf) {
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int c = tid + 512 * q, kk = c >> 6, c4 = 4 * (c & 63);
      put(&sm[buf][0], kk, c4, rp[q]);
      put(&sm[buf][3 * PLANE], kk, c4, rq[q]);
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
  load(0);
  store(0);
  __syncthreads();
  for (int kc = 0; kc < nk; ++kc) {
    const int cur = kc & 1;
    if (kc + 1 < nk) load((kc + 1) * kX6BK);
    bf16x8_t fa[3][NBM], fb[3][NBN];
#pragma unroll
    for (int t = 0; t < 3; ++t) {
#pragma unroll
      for (int a = 0; a < NBM; ++a) fa[t][a] = frag32_tr(&sm[cur][t * PLANE], LD, wi * WM + 32 * a, 0, lane);
#pragma unroll
      for (int b = 0; b < NBN; ++b) fb[t][b] = frag32_tr(&sm[cur][(3 + t) * PLANE], LD, wj * WN + 32 * b, 0, lane);
    }
    // the six kept terms, smallest first; each term runs over all blocks, so the MFMAs
    // into one accumulator are eight instructions apart
    constexpr int TA[6] = {2, 0, 1, 1, 0, 0}, TB[6] = {0, 2, 1, 0, 1, 0};
#pragma unroll
    for (int t = 0; t < 6; ++t)
#pragma unroll
      for (int a = 0; a < NBM; ++a)
#pragma unroll
        for (int b = 0; b < NBN; ++b) acc[a][b] = mfma32(fa[TA[t]][a], fb[TB[t]][b], acc[a][b]);
    if (kc + 1 < nk) store(cur ^ 1);
    __syncthreads();
  }
  if (!active) return;
#pragma unroll
  for (int a = 0; a < NBM; ++a)
#pragma unroll
    for (int b = 0; b < NBN; ++b) {
      const int64_t col = ocol + wj * WN + 32 * b + mfma32_col(lane);
      const int64_t rb = orow + wi * WM + 32 * a;
      float old[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t row = rb + mfma32_row(lane, r);
        old[r] = ld_or_zero(F, row * d + col, row < d && col < d && col >= row);
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t row = rb + mfma32_row(lane, r);
        if (row < d && col < d && col >= row) F[row * d + col] = old[r] - acc[a][b][r];
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
  // Blocked right-looking factorization with the forward substitution of the RHS
  // carried along.  The trailing matrix is updated once per super-panel of kSuper
  // panels (one pass over it per kSuper * P columns); inside a super-panel each panel
  // first receives the contributions of the super-panel's earlier panels (a strip
  // update of its own rows), then is factored (diagonal block) and solved (row panel).
  constexpr int P = Mf<T>::P, kSuper = 4;
  const bool x6 = sizeof(T) == 4 && d % 4 == 0;
  const int64_t TM = (m + P - 1) / P;
  for (int64_t P0 = 0; P0 < d; P0 += kSuper * P) {
    const int64_t P1 = (d - P0) < kSuper * P ? d : P0 + kSuper * P;
    for (int64_t pp = P0; pp < P1; pp += P) {
      const int64_t pw = (d - pp) < P ? (d - pp) : P;
      const int64_t nrem = d - pp - pw;
      if (pp > P0) {
        const int64_t T2 = (d - pp + P - 1) / P;
        k_panel_product<T, kTrailing><<<dim3((unsigned)(T2 + TM), (unsigned)nm), kT, 0, a.stream>>>(
            d, m, 0, P0, pp - P0, pp, 1, 0, F, R);
      }
      k_diag_block<T><<<(unsigned)nm, kT, 0, a.stream>>>(d, pp, F, a.dev_info);
      const int64_t nch = (nrem + P - 1) / P + TM;
      k_panel_product<T, kRowPanel><<<dim3((unsigned)nch, (unsigned)nm), kT, 0, a.stream>>>(d, m, pp, 0, 0, 0, 0, 0,
                                                                                             F, R);
    }
    if (P1 < d) {
      const int64_t T2 = (d - P1 + P - 1) / P, nU = T2 * (T2 + 1) / 2;
      if (x6) {
        const int64_t T6 = (d - P1 + 255) / 256;
        k_trail_x6<<<dim3((unsigned)(T6 * (T6 + 1) / 2), (unsigned)nm), 512, 0, a.stream>>>(d, P0, P1 - P0, P1,
                                                                                            (float*)F);
        k_panel_product<T, kTrailing><<<dim3((unsigned)(T2 * TM), (unsigned)nm), kT, 0, a.stream>>>(
            d, m, 0, P0, P1 - P0, P1, 0, (int)nU, F, R);
      } else {
        k_panel_product<T, kTrailing><<<dim3((unsigned)(nU + T2 * TM), (unsigned)nm), kT, 0, a.stream>>>(
            d, m, 0, P0, P1 - P0, P1, 0, 0, F, R);
      }
    }
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  for (int64_t pp = ((d - 1) / P) * P; pp >= 0; pp -= P) {
    const dim3 grid((unsigned)(pp > 0 ? (pp + P - 1) / P : 1), (unsigned)nm);
    const int nq = (int)((m + Mf<T>::BLK - 1) / Mf<T>::BLK);  // m <= 128 (checked by the API)
    if (nq <= 1) k_back_step<T, 1><<<grid, kT, 0, a.stream>>>(d, m, pp, F, R, Mp);
    else if (nq <= 2) k_back_step<T, 2><<<grid, kT, 0, a.stream>>>(d, m, pp, F, R, Mp);
    else if (nq <= 4 || sizeof(T) == 4) k_back_step<T, 4><<<grid, kT, 0, a.stream>>>(d, m, pp, F, R, Mp);
    else if constexpr (sizeof(T) == 8) k_back_step<T, 8><<<grid, kT, 0, a.stream>>>(d, m, pp, F, R, Mp);
  }
  k_unscale<T><<<dim3((unsigned)((d * m + 255) / 256), (unsigned)nm), 256, 0, a.stream>>>(d, m, Mp, D, a.m_out,
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
