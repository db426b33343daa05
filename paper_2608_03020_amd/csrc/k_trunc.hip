// k_trunc.hip -- rank-r_a truncation (row a6) and the paper's projected fit (row a5, Eqs. 6-9).
//
// Truncation (Lemma S5.2, Eckart-Young) of W = M R with M: d x kp, R: kp x d,
// without forming W: with the small Gram matrices Gm = M^T M, Gb = R R^T
// (kp x kp, fp64) and Gb = Vb diag(lb) Vb^T, H = diag(sqrt(lb)),
//   W = (M Vb H)(H^{-1} Vb^T R)  where H^{-1} Vb^T R has orthonormal rows,
// so the singular values of W are those of P = M Vb H, whose right factor
// comes from the eigendecomposition H Vb^T Gm Vb H = Vp diag(s^2) Vp^T.  Then
//   U = M Vb H Vp diag(1/s),   V = R^T Vb H^{-1} Vp,
//   a_out = U_r^T = Ca M^T,    b_out = V_r diag(s_r) = R^T Cb
// with small Ca (r x kp) and Cb (kp x r).  Both eigendecompositions are
// cyclic Jacobi in fp64 inside one workgroup, the symmetric matrix packed in LDS:
// for kp <= 64 with the eigenvectors and the kp x kp intermediates in LDS (fp64);
// for 64 < kp <= 128 with the eigenvectors in LDS as floats (rotations computed in
// fp64) and the kp x kp intermediates in the workspace.
#include "loca_launch.h"

namespace loca {

namespace {

constexpr int kT = 256;
constexpr int kMaxKp = 64;
constexpr int kMaxKpBig = 128;
constexpr int kMaxRank = 64;  // r_a

// Partial Gm = M^T M and Gb = R R^T (fp64) over the row range of blockIdx.z (of nsplit
// equal ranges of 32-row multiples); blockIdx.x = matrix, blockIdx.y = 0 (M) / 1 (R).
// The partials are summed in a fixed order by k_trunc_core.  Each 32-row chunk is staged
// in LDS as doubles (the next one is loaded into registers meanwhile) and its products
// are formed on the fp64 matrix cores (v_mfma_f64_16x16x4f64; products of floats are
// exact in fp64): the kp x kp result is cut into 16 x 16 blocks, wave w taking the
// blocks w, w + 4, ...
template <int KPM>
__global__ __launch_bounds__(kT) void k_small_grams(int64_t d, int64_t kp, const float* __restrict__ M,
                                                    int64_t m_bstride, const float* __restrict__ R,
                                                    int64_t r_bstride, int64_t r_group, int nsplit,
                                                    double* __restrict__ Gpart) {
  constexpr int kRows = 32;
  constexpr int kLd = KPM + 1;
  constexpr int kPer = kRows * KPM / kT;                // staged values per thread and chunk, at most
  constexpr int kBlk = (KPM / 16) * (KPM / 16) / 4;     // output blocks per wave, at most
  __shared__ double sX[kRows * kLd];
  const int64_t mi = blockIdx.x;
  const bool isR = blockIdx.y == 1;
  const int64_t chunk = ((d + nsplit - 1) / nsplit + kRows - 1) / kRows * kRows;
  const int64_t ib = (int64_t)blockIdx.z * chunk, ie = ib + chunk < d ? ib + chunk : d;
  const float* Mm = M + mi * m_bstride;
  const float* Rm = R + (mi / r_group) * r_bstride;
  const int K = (int)kp, nb = (K + 15) / 16, nv = kRows * K;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, kr = lane >> 4, cr = lane & 15;
  // staged element f of a chunk: (row, column) (R's rows are contiguous along i)
  auto where = [&](int f) { return isR ? make_int2(f % kRows, f / kRows) : make_int2(f / K, f % K); };
  for (int e = tid; e < kRows * kLd; e += kT) sX[e] = 0.0;  // columns past kp stay zero
  float v[kPer];
  auto load = [&](int64_t i0) {
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const int f = tid + kT * j;
      float x = 0.f;
      if (f < nv) {
        const int2 rc = where(f);
        const int64_t i = i0 + rc.x;
        if (i < ie) x = isR ? Rm[rc.y * d + i] : Mm[i * kp + rc.y];
      }
      v[j] = x;
    }
  };
  f64x4_t acc[kBlk];
#pragma unroll
  for (int q = 0; q < kBlk; ++q) acc[q] = f64x4_t{0.0, 0.0, 0.0, 0.0};
  if (ib < ie) load(ib);
  for (int64_t i0 = ib; i0 < ie; i0 += kRows) {
    __syncthreads();  // the previous chunk is no longer read (and the zero fill is done)
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const int f = tid + kT * j;
      if (f < nv) {
        const int2 rc = where(f);
        sX[rc.x * kLd + rc.y] = (double)v[j];
      }
    }
    __syncthreads();
    if (i0 + kRows < ie) load(i0 + kRows);
#pragma unroll
    for (int q = 0; q < kBlk; ++q) {
      const int blk = w + 4 * q;
      if (blk < nb * nb) {  // A[i][x] = X[x][ba + i], B[x][j] = X[x][bc + j]
        const int ba = 16 * (blk / nb), bc = 16 * (blk % nb);
#pragma unroll
        for (int kk = 0; kk < kRows; kk += 4)
          acc[q] = mfma_f64(sX[(kk + kr) * kLd + ba + cr], sX[(kk + kr) * kLd + bc + cr], acc[q]);
      }
    }
  }
  double* G = Gpart + ((mi * 2 + (isR ? 1 : 0)) * nsplit + blockIdx.z) * kp * kp;
#pragma unroll
  for (int q = 0; q < kBlk; ++q) {
    const int blk = w + 4 * q;
    if (blk < nb * nb) {
      const int ba = 16 * (blk / nb), bc = 16 * (blk % nb);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = ba + kr + 4 * r, col = bc + cr;
        if (row < K && col < K) G[row * kp + col] = acc[q][r];
      }
    }
  }
}

// Threads of the eigensolver workgroups (one workgroup per matrix): sixteen waves, four per
// SIMD, so that the waves hide each other's LDS latency in the rounds of the Jacobi
// iteration, whose updates are chains of dependent LDS reads and writes.
constexpr int kTC = 1024;
// the workgroup's reduction scratch (doubles): two block sums, then flags and scalars
constexpr int kRedSum0 = 0, kRedSum1 = 16, kRedConv = 32, kRedRot = 33, kRedMax = 40, kRedDiag = 41,
              kRedFail = 42, kRedLen = 48;

// ------------------------------------------------------------------ symmetric eigensolver

// Upper-triangle packed index of (i, j) in either order, n x n.
LOCA_DEV int pk(int i, int j, int n) {
  if (i > j) { const int t = i; i = j; j = t; }
  return i * n - (i * (i - 1)) / 2 + (j - i);
}

// 1/x and 1/sqrt(x) in double from the hardware approximations and two Newton steps each
// (full double precision for the finite, nonzero arguments of the rotations below).
LOCA_DEV double rcp64(double x) {
  double y = __builtin_amdgcn_rcp(x);
#pragma unroll
  for (int i = 0; i < 2; ++i) y = fma(y, fma(-x, y, 1.0), y);
  return y;
}
// 1/x from the hardware approximation and one Newton step (about 2^-46 relative).
LOCA_DEV double rcp64_1(double x) {
  const double y = __builtin_amdgcn_rcp(x);
  return fma(y, fma(-x, y, 1.0), y);
}
LOCA_DEV double rsq64(double x) {
  double y = __builtin_amdgcn_rsq(x);
#pragma unroll
  for (int i = 0; i < 2; ++i) y = y * fma(-0.5 * x * y, y, 1.5);
  return y;
}

// Cyclic Jacobi on the packed symmetric n x n matrix A (n even), eigenvectors into the
// n x n V of type VT (row-major, columns are the vectors; rotations computed in fp64).  Each
// round rotates n/2 disjoint pairs (round-robin tournament order: position 0 fixed, the
// others rotating, so that a sweep of n - 1 rounds meets every pair once) as
// one two-sided update: every 2 x 2 block of rows {p_k, q_k} and columns {p_l, q_l} is
// owned by one thread and becomes J_k^T B J_l.  A pair is rotated while
// a_pq^2 > 1e-30 |a_pp a_qq| (|a_pq| above 1e-15 of the geometric mean of its diagonal
// entries); the iteration ends after a sweep that rotates nothing, or once the
// off-diagonal part is below 1e-30 of the squared Frobenius norm.  While the rotations
// run, V holds the vectors as rows, so that a rotation combines two contiguous rows with
// the lanes along them (no LDS bank conflicts); it is transposed at the end.  A pair is
// read as one int2 and its (c, s) as one double2 (`pairs`, `cs` 16-byte aligned).  Run by
// the kTC threads of one workgroup; `red` holds kRedLen doubles.
template <typename VT>
LOCA_DEV void jacobi_packed(double* A, VT* V, int n, double* cs, int* pairs, double* red) {
  const int tid = threadIdx.x, m = n / 2;
  const int2* pr = (const int2*)pairs;
  const double2* cs2 = (const double2*)cs;
  for (int e = tid; e < n * n; e += kTC) V[e] = ((e / n) == (e % n)) ? (VT)1 : (VT)0;
  __syncthreads();
  for (int sweep = 0; sweep < 40; ++sweep) {
    double off = 0.0, tot = 0.0;
    for (int e = tid; e < n * n; e += kTC) {
      const int i = e / n, j = e % n;
      const double v = A[pk(i, j, n)];
      tot += v * v;
      if (i != j) off += v * v;
    }
    const double offs = block_sum(off, red + kRedSum0);
    __syncthreads();
    const double tots = block_sum(tot, red + kRedSum1);
    if (tid == 0) {
      red[kRedConv] = (offs <= 1e-30 * tots || tots == 0.0) ? 1.0 : 0.0;
      red[kRedRot] = 0.0;  // set by any rotation of this sweep
    }
    __syncthreads();
    if (red[kRedConv] != 0.0) break;
    for (int round = 0; round < n - 1; ++round) {
      if (tid < m) {
        auto pos = [&](int x) { return x == 0 ? 0 : 1 + ((x - 1 + round) % (n - 1)); };
        int p = pos(tid), q = pos(n - 1 - tid);
        if (p > q) { const int t = p; p = q; q = t; }
        ((int2*)pairs)[tid] = make_int2(p, q);
        const double apq = A[pk(p, q, n)], app = A[pk(p, p, n)], aqq = A[pk(q, q, n)];
        double c = 1.0, s = 0.0;
        if (fabs(apq) > 1e-300 && apq * apq > 1e-30 * fabs(app * aqq)) {
          const double tau = (aqq - app) * rcp64(2.0 * apq);
          const double u = 1.0 + tau * tau;
          const double t = (tau >= 0.0 ? 1.0 : -1.0) * rcp64(fabs(tau) + u * rsq64(u));
          c = rsq64(1.0 + t * t);
          s = t * c;
          red[kRedRot] = 1.0;
        }
        ((double2*)cs)[tid] = make_double2(c, s);
      }
      __syncthreads();
      for (int e = tid; e < m * m; e += kTC) {
        const int k = e / m, l = e % m;
        if (k > l) continue;
        const int2 qk = pr[k], ql = pr[l];
        const double2 rk = cs2[k], rl = cs2[l];
        const double ck = rk.x, sk = rk.y, cl = rl.x, sl = rl.y;
        const double b00 = A[pk(qk.x, ql.x, n)], b01 = A[pk(qk.x, ql.y, n)];
        const double b10 = A[pk(qk.y, ql.x, n)], b11 = A[pk(qk.y, ql.y, n)];
        const double x00 = cl * b00 - sl * b01, x01 = sl * b00 + cl * b01;  // B J_l
        const double x10 = cl * b10 - sl * b11, x11 = sl * b10 + cl * b11;
        const double y00 = ck * x00 - sk * x10, y01 = ck * x01 - sk * x11;  // J_k^T B J_l
        const double y10 = sk * x00 + ck * x10, y11 = sk * x01 + ck * x11;
        if (k == l) {
          A[pk(qk.x, qk.x, n)] = y00;
          A[pk(qk.y, qk.y, n)] = y11;
          A[pk(qk.x, qk.y, n)] = 0.0;
        } else {
          A[pk(qk.x, ql.x, n)] = y00;
          A[pk(qk.x, ql.y, n)] = y01;
          A[pk(qk.y, ql.x, n)] = y10;
          A[pk(qk.y, ql.y, n)] = y11;
        }
      }
      for (int e = tid; e < n * m; e += kTC) {  // rows p, q of V^T: V^T <- J^T V^T
        const int k = e / n, i = e % n;
        const int2 q2 = pr[k];
        const double2 r = cs2[k];
        const double vp = V[q2.x * n + i], vq = V[q2.y * n + i];
        V[q2.x * n + i] = (VT)(r.x * vp - r.y * vq);
        V[q2.y * n + i] = (VT)(r.y * vp + r.x * vq);
      }
      __syncthreads();
    }
    if (red[kRedRot] == 0.0) break;  // a whole sweep found every pair below the threshold
  }
  for (int e = tid; e < n * n; e += kTC) {  // the vectors from rows to columns
    const int i = e / n, j = e % n;
    if (i < j) {
      const VT x = V[i * n + j], y = V[j * n + i];
      V[i * n + j] = y;
      V[j * n + i] = x;
    }
  }
  __syncthreads();
}

// ------------------------------------------------------------------ symmetric eigensolver, leading part

// A double moved between lanes of a row of 16 by a DPP pattern (CTRL: quad_perm or row_ror).
template <int CTRL>
LOCA_DEV double dpp_d(double v) {
  const long long b = __double_as_longlong(v);
  const int lo = __builtin_amdgcn_update_dpp(0, (int)b, CTRL, 0xF, 0xF, false);
  const int hi = __builtin_amdgcn_update_dpp(0, (int)(b >> 32), CTRL, 0xF, 0xF, false);
  return __longlong_as_double(((long long)hi << 32) | (long long)(unsigned)lo);
}
// Sum over aligned groups of 16 lanes by DPP moves (quad xor 1 and 2, then row rotations by
// 4 and 8); every lane of a group gets the sum, possibly differing in the last bit between
// its quads (the two rotations associate the four quad sums differently).
LOCA_DEV double seg16_sum(double v) {
  v += dpp_d<0xB1>(v);   // quad_perm [1,0,3,2]
  v += dpp_d<0x4E>(v);   // quad_perm [2,3,0,1]
  v += dpp_d<0x124>(v);  // row_ror:4
  v += dpp_d<0x128>(v);  // row_ror:8
  return v;
}
// Sum over aligned groups of 8 lanes (quad xor 1 and 2, then the half-row mirror).
LOCA_DEV double seg8_sum(double v) {
  v += dpp_d<0xB1>(v);   // quad_perm [1,0,3,2]
  v += dpp_d<0x4E>(v);   // quad_perm [2,3,0,1]
  v += dpp_d<0x141>(v);  // row_half_mirror
  return v;
}
LOCA_DEV double readlane_d(double v, int l) {
  const long long b = __double_as_longlong(v);
  const int lo = __builtin_amdgcn_readlane((int)b, l);
  const int hi = __builtin_amdgcn_readlane((int)(b >> 32), l);
  return __longlong_as_double(((long long)hi << 32) | (long long)(unsigned)lo);
}
// Sum over the lanes of a wave: the sums of the four rows of 16, then their total in a
// fixed order from lanes 0, 16, 32, 48, the same value in every lane (and in every wave
// that sums the same data).
LOCA_DEV double wave_sum_all(double v) {
  v = seg16_sum(v);
  return (readlane_d(v, 0) + readlane_d(v, 16)) + (readlane_d(v, 32) + readlane_d(v, 48));
}
// A pivot of magnitude below pivmin is replaced by -pivmin (a Sturm count then treats it as
// negative, and no quotient overflows).
LOCA_DEV double safe_pivot(double q, double pivmin) { return fabs(q) < pivmin ? -pivmin : q; }

constexpr int kRedEig = 43;   // reduction-scratch slot: a check of eig_top failed
constexpr int kRedLive = 44;  // ... the number of pairs eig_top returned

// All eigenvalues of the packed symmetric K x K matrix A (packed with stride n, K <= KM) and
// the eigenvectors of its r largest, A left unchanged:
//   1. Householder reduction T = Q^T A Q to tridiagonal form on the working matrix W (a
//      dense copy of A, or, PACKED, A's packed triangle in place), two barriers per step:
//      every wave forms the reflector v of row k itself, p = tau A v with kTC / KM lanes per
//      row, then every wave w = p - (tau/2)(p^T v) v and the rank-2 update
//      A -= v w^T + w v^T over a 32 x 32 grid of threads; the reflector is stored in row k
//      right of the diagonal;
//   2. every eigenvalue of T by multisection of Sturm counts: L = kTC / KM lanes per
//      eigenvalue test the L - 1 interior points of L equal steps of its interval; for the r
//      largest until the widened Gershgorin interval (at most 2.2 ||T||) has shrunk 2^52
//      times or more, a few units of double rounding of ||T||, the accuracy of the Sturm
//      counts themselves; 2^40 for the others, whose only use is the float sigma; the
//      pivots' reciprocals from the hardware approximation and one Newton step;
//   3. the eigenvector of T for each of the r largest (one lane each) from the twisted
//      factorization of T - lambda I: the pivots of the top-down and bottom-up LDL^T, the
//      twist index where their combination is smallest, and one solve that starts there;
//   4. x = Q z (the reflectors applied in reverse order; 16 lanes per vector), stored in
//      column j < r of Vout (row-major, stride n, type OutT); the other entries are zero.
// Only eigenvalues above 1e-12 ||T|| (one Sturm count) get vectors: r is lowered to their
// number when A has rank below r (its numerical zeros among the r largest have no
// separable vectors, and their directions carry no weight), and lowered again to j when
// eigenvalues j and j + 1 (both among the r largest) lie within 1e-10 of the largest
// |lambda| of each other and |lambda_j| does of zero (numerical zeros above that count, as
// left by the rounding of float factors); the count is left in red[kRedLive].  The path is
// left (false returned, and the caller runs Jacobi on A) before the vectors when two other
// of the r largest lie that close (a repeated value), and after them when the check fails: every residual
// ||A x - lambda x|| and every pair of the r vectors orthonormal within 1e-11 and 1e-9
// (float vectors: 1e-5 and 1e-5).  On success eig[j] is the j-th largest eigenvalue
// (j < K).  Z: r x K doubles of scratch (it may share Vout's memory); dT, eT, e2, tauH,
// pbuf: KM doubles each.  Run by the kTC threads of one workgroup.
template <int KM, bool PACKED, typename OutT>
LOCA_DEV bool eig_top(const double* A, int n, int K, int r, double* W, OutT* Vout, double* Z, double* dT,
                      double* eT, double* e2, double* tauH, double* pbuf, double* eig, double* red) {
  static_assert(KM == 64 || KM == 128, "workgroup maps for K <= 64 or K <= 128");
  constexpr int LPR = kTC / KM;  // lanes per row of p, and per eigenvalue in the multisection
  constexpr int NX = KM / 64, NP = KM / LPR, NU = KM / 32, NZ = KM / 16;
  const int tid = threadIdx.x, lane = tid & 63;
  auto at = [&](int i, int j) -> double& { return PACKED ? W[pk(i, j, n)] : W[i * n + j]; };
  auto segsum = [&](double v) { return LPR == 16 ? seg16_sum(v) : seg8_sum(v); };
  if (!PACKED)
    for (int e = tid; e < n * n; e += kTC) {
      const int i = e / n, j = e % n;
      W[e] = (i < K && j < K) ? A[pk(i, j, n)] : 0.0;
    }
  __shared__ int s_cut;  // the number of pairs while it is lowered
  int* cut = &s_cut;
  if (tid == 0) red[kRedEig] = 0.0;
  __syncthreads();
  // 1. reduction to tridiagonal form
  {
    const int ty = tid >> 5, tx = tid & 31;
    for (int k = 0; k + 2 < K; ++k) {
      const int m = K - k - 1;  // entries right of the diagonal in row k
      // the reflector of row k, formed by every wave alike (row k is final since the
      // last barrier); row k keeps x until the step's end, v_0 is kept apart
      double xs[NX];
      double sq = 0.0;
#pragma unroll
      for (int u = 0; u < NX; ++u) {
        const int c = lane + 64 * u;
        xs[u] = c < m ? at(k, k + 1 + c) : 0.0;
        sq += xs[u] * xs[u];
      }
      const double ss = wave_sum_all(sq);
      const double x0 = at(k, k + 1);
      double tau = 0.0, alpha = x0, v0 = x0;
      if (ss > 0.0) {
        const double nx = ss > 1e-280 ? ss * rsq64(ss) : sqrt(ss);  // ||x||
        alpha = x0 >= 0.0 ? -nx : nx;
        v0 = x0 - alpha;
        tau = 2.0 * rcp64(ss - x0 * x0 + v0 * v0);
      }
      if (tid == 0) {
        tauH[k] = tau;
        eT[k] = alpha;
        dT[k] = at(k, k);
      }
      if (tau != 0.0) {  // uniform: every wave has the same ss
        {  // p_i = tau sum_c A[k+1+i][k+1+c] v_c, LPR lanes per row i
          const int row = tid / LPR, part = tid % LPR;
          double acc = 0.0;
          if (row < m)
#pragma unroll
            for (int u = 0; u < NP; ++u) {
              const int c = part + LPR * u;
              if (c < m) acc += at(k + 1 + row, k + 1 + c) * (c == 0 ? v0 : at(k, k + 1 + c));
            }
          acc = segsum(acc);
          if (row < m && part == 0) pbuf[row] = tau * acc;
        }
        __syncthreads();
        double pv = 0.0;
#pragma unroll
        for (int u = 0; u < NX; ++u) {
          const int c = lane + 64 * u;
          if (c < m) pv += pbuf[c] * (c == 0 ? v0 : xs[u]);
        }
        const double kk = 0.5 * tau * wave_sum_all(pv);
        // A[k+1+i][k+1+c] -= v_i w_c + w_i v_c, w = p - kk v (upper triangle only when
        // packed); thread (ty, tx) takes i in {ty + 32 a}, c in {tx + 32 b}
#pragma unroll
        for (int a = 0; a < NU; ++a) {
          const int i = ty + 32 * a;
          if (i >= m) continue;
          const double vi = i == 0 ? v0 : at(k, k + 1 + i);
          const double wi = pbuf[i] - kk * vi;
#pragma unroll
          for (int b = 0; b < NU; ++b) {
            const int c = tx + 32 * b;
            if (c >= m || (PACKED && c < i)) continue;
            const double vc = c == 0 ? v0 : at(k, k + 1 + c);
            const double wc = pbuf[c] - kk * vc;
            at(k + 1 + i, k + 1 + c) -= vi * wc + wi * vc;
          }
        }
      }
      __syncthreads();
      if (tid == 0) at(k, k + 1) = v0;  // the reflector complete in row k (read only later)
    }
    if (tid == 0) {
      if (K >= 2) {
        dT[K - 2] = at(K - 2, K - 2);
        eT[K - 2] = at(K - 2, K - 1);
      }
      dT[K - 1] = at(K - 1, K - 1);
    }
  }
  __syncthreads();
  for (int i = tid; i + 1 < K; i += kTC) e2[i] = eT[i] * eT[i];
  // Gershgorin interval, widened as in LAPACK's bisection, and the pivot floor
  double glo = 0.0, ghi = 0.0, emax2 = 0.0;
  for (int i = 0; i < K; ++i) {
    const double rad = (i > 0 ? fabs(eT[i - 1]) : 0.0) + (i + 1 < K ? fabs(eT[i]) : 0.0);
    glo = i == 0 ? dT[i] - rad : fmin(glo, dT[i] - rad);
    ghi = i == 0 ? dT[i] + rad : fmax(ghi, dT[i] + rad);
    if (i + 1 < K) emax2 = fmax(emax2, eT[i] * eT[i]);
  }
  const double pivmin = 2.2250738585072014e-308 * fmax(1.0, emax2);
  const double tnorm = fmax(fabs(glo), fabs(ghi));
  glo -= 2.1 * tnorm * 2.220446049250313e-16 * K + 4.2 * pivmin;
  ghi += 2.1 * tnorm * 2.220446049250313e-16 * K + 4.2 * pivmin;
  __syncthreads();
  const int r_req = r;  // the pairs asked for: their eigenvalues all get the full precision
  {  // only the eigenvalues above 1e-12 ||T|| get vectors: below it the r largest would hold
     // a cluster of numerical zeros (A of rank below r), whose vectors the twisted solves
     // cannot separate and whose directions carry no weight (every thread counts alike)
    const double x0 = 1e-12 * tnorm;
    double q = safe_pivot(dT[0] - x0, pivmin);
    int below = q < 0.0;
    for (int i = 1; i < K; ++i) {
      q = safe_pivot((dT[i] - x0) - e2[i - 1] * rcp64_1(q), pivmin);
      below += q < 0.0;
    }
    if (K - below < r) r = K - below;
    if (tid == 0) *cut = r;
  }
  // 2. multisection: group g = tid / LPR finds the g-th smallest eigenvalue, lane t of the
  // group testing point t + 1 of LPR equal steps (the last one is hi); for the r largest
  // asked for (whose vectors follow, and whose singular values are reported to the same
  // accuracy when they are numerical zeros), 52 bits or more of the interval (13 steps of
  // 16, 18 of 8), for the others 40 or more (10 of 16, 14 of 8)
  {
    constexpr int STEPS_V = LPR == 16 ? 13 : 18, STEPS_S = LPR == 16 ? 10 : 14;
    const int g = tid / LPR, t = tid % LPR;
    const int j = g < K ? g : K - 1;
    const int steps = K - 1 - j < r_req ? STEPS_V : STEPS_S;
    double lo = glo, hi = ghi;
    for (int it = 0; it < steps; ++it) {
      const double h = (hi - lo) * (1.0 / LPR);
      const double x = lo + (double)(t + 1) * h;
      double q = safe_pivot(dT[0] - x, pivmin);
      int cnt = q < 0.0;
      for (int i = 1; i < K; ++i) {
        q = safe_pivot((dT[i] - x) - e2[i - 1] * rcp64_1(q), pivmin);
        cnt += q < 0.0;
      }
      if (t == LPR - 1) cnt = K;
      const unsigned long long b = __ballot(cnt > j);
      const unsigned seg = (unsigned)(b >> (lane & (64 - LPR))) & ((1u << LPR) - 1u);  // last lane set
      const int f = __builtin_ctz(seg);
      const double nlo = f == 0 ? lo : lo + (double)f * h;
      hi = f == LPR - 1 ? hi : lo + (double)(f + 1) * h;
      lo = nlo;
    }
    if (g < K && t == 0) eig[K - 1 - g] = 0.5 * (lo + hi);
  }
  __syncthreads();
  // eigenvalues among the r largest closer than 1e-10 of the largest |lambda| (a repeated
  // value) cannot get orthogonal vectors from the twisted solves: Jacobi at once
  {
    const double sc = fmax(fabs(eig[0]), fabs(eig[K - 1]));
    if (tid + 1 < r && !(eig[tid] - eig[tid + 1] > 1e-10 * sc)) {
      if (fabs(eig[tid]) <= 1e-10 * sc)
        atomicMin(cut, tid);  // numerical zeros: no vectors from the first of them on
      else
        red[kRedEig] = 1.0;
    }
  }
  __syncthreads();
  if (red[kRedEig] != 0.0) return false;
  r = *cut;
  if (tid == 0) red[kRedLive] = (double)r;
  // 3. twisted factorizations (lane a: the a-th largest eigenvalue; scratch row Z + a K)
  if (tid < r) {
    const double lam = eig[tid];
    double* w = Z + tid * K;
    double dp = safe_pivot(dT[0] - lam, pivmin);
    w[0] = dp;
    for (int i = 0; i + 1 < K; ++i) {
      dp = safe_pivot((dT[i + 1] - lam) - e2[i] * rcp64(dp), pivmin);
      w[i + 1] = dp;
    }
    double dm = safe_pivot(dT[K - 1] - lam, pivmin);
    int rr = K - 1;
    double gmin = fabs(w[K - 1]);
    for (int i = K - 2; i >= 0; --i) {
      const double u = eT[i] * rcp64(dm);
      const double dmi = safe_pivot((dT[i] - lam) - u * eT[i], pivmin);
      const double gam = w[i] + dmi - (dT[i] - lam);
      if (fabs(gam) < gmin) {
        gmin = fabs(gam);
        rr = i;
      }
      w[i] = u;  // u_i replaces the top-down pivot
      dm = dmi;
    }
    double z = 1.0, nrm = 1.0;
    for (int i = rr; i + 1 < K; ++i) {  // z_{i+1} = -u_i z_i
      const double u = w[i];
      w[i] = z;
      z = -u * z;
      nrm += z * z;
    }
    w[K - 1] = z;
    if (rr > 0) {  // z_i = -l_i z_{i+1} with l_i = e_i / (top-down pivot i), recomputed
      double dq = safe_pivot(dT[0] - lam, pivmin);
      for (int i = 0; i < rr; ++i) {
        const double l = eT[i] * rcp64(dq);
        w[i] = l;
        dq = safe_pivot((dT[i + 1] - lam) - l * eT[i], pivmin);
      }
      double zz = 1.0;
      for (int i = rr - 1; i >= 0; --i) {
        zz = -w[i] * zz;
        w[i] = zz;
        nrm += zz * zz;
      }
    }
    const double sc = rsq64(nrm);
    for (int i = 0; i < K; ++i) w[i] *= sc;
  }
  __syncthreads();
  // 4. x = H_0 H_1 ... H_{K-3} z: 16 lanes per vector, entries t + 16 q in registers
  {
    const int a = tid >> 4, t = tid & 15;
    const bool act = a < r;
    double zr[NZ];
#pragma unroll
    for (int q = 0; q < NZ; ++q) {
      const int i = t + 16 * q;
      zr[q] = (act && i < K) ? Z[a * K + i] : 0.0;
    }
    for (int k = K - 3; k >= 0; --k) {
      const double tau = tauH[k];
      if (tau == 0.0) continue;
      double dot = 0.0;
#pragma unroll
      for (int q = 0; q < NZ; ++q) {
        const int i = t + 16 * q;
        if (i > k && i < K) dot += at(k, i) * zr[q];
      }
      const double f = tau * seg16_sum(dot);
#pragma unroll
      for (int q = 0; q < NZ; ++q) {
        const int i = t + 16 * q;
        if (i > k && i < K) zr[q] -= f * at(k, i);
      }
    }
    __syncthreads();  // the reflectors and Z are read by every group before Vout is written
    for (int e = tid; e < n * n; e += kTC) {
      const int i = e / n, j = e % n;
      if (j >= r || i >= K) Vout[e] = (OutT)0;
    }
    if (act)
#pragma unroll
      for (int q = 0; q < NZ; ++q) {
        const int i = t + 16 * q;
        if (i < K) Vout[i * n + a] = (OutT)zr[q];
      }
  }
  __syncthreads();
  // the check (vectors as stored: a float copy is held to float accuracy)
  constexpr double kRes = sizeof(OutT) == 8 ? 1e-11 : 1e-5, kOrth = sizeof(OutT) == 8 ? 1e-9 : 1e-5;
  const double anorm = fmax(fabs(eig[0]), fabs(eig[K - 1]));
  {
    const int a = tid >> 4, t = tid & 15;
    double rs = 0.0;
    if (a < r) {
      const double lam = eig[a];
      for (int i = t; i < K; i += 16) {
        double s = -lam * (double)Vout[i * n + a];
        for (int c = 0; c < K; ++c) s += A[pk(i, c, n)] * (double)Vout[c * n + a];
        rs += s * s;
      }
    }
    rs = seg16_sum(rs);
    const double tol = kRes * anorm;
    if (a < r && t == 0 && !(rs <= tol * tol)) red[kRedEig] = 1.0;
  }
  for (int e = tid; e < r * r; e += kTC) {
    const int a = e / r, b = e % r;
    if (a > b) continue;
    double s = 0.0;
    for (int i = 0; i < K; ++i) s += (double)Vout[i * n + a] * (double)Vout[i * n + b];
    if (!(fabs(s - (a == b ? 1.0 : 0.0)) <= kOrth)) red[kRedEig] = 1.0;
  }
  __syncthreads();
  return red[kRedEig] == 0.0;
}

// The truncation core for 64 < kp <= 128 (see the file comment).  As the core for kp <= 64:
// Gb = R R^T = U^T U by Cholesky when every pivot exceeds 1e-10 of the largest diagonal
// entry (then W = (M L)(L^{-1} R) with L = U^T, one eigensolve of P^T P = L^T Gm L, and
// Ca[a][c] = (L Vp)[c][a] / s_a, Cb[c][a] = (L^{-T} Vp)[c][a] s_a), otherwise the
// eigendecomposition of Gb by Jacobi and H as in the file comment.  The packed symmetric
// matrix of the eigensolve lives in LDS; its kept pairs come from the tridiagonal path
// (eig_top, reduced in place, the vectors stored as floats), Jacobi taking over (the
// eigenvectors in LDS as floats, rotations in fp64) when its check fails.  Per matrix the workspace `big` holds two n x n fp64 matrices (n = kp rounded up to
// even): Gm (then Gm L, then L^{-T} Vp) and L (or T = Gm Vb), from big + mi * 2 kMaxKpBig^2
// doubles, then after nm such pairs a float copy of Vb per matrix.
__global__ __launch_bounds__(kTC) void k_trunc_core_big(int64_t nm, int64_t kp, int64_t r_a,
                                                        const double* __restrict__ Gpart, int nsplit,
                                                        double* __restrict__ big, double* __restrict__ Ca_all,
                                                        double* __restrict__ Cb_all, float* __restrict__ sigma_out,
                                                        int64_t sigma_bstride, int32_t* __restrict__ live_out) {
  constexpr int KB2 = kMaxKpBig * kMaxKpBig;
  __shared__ double sA[kMaxKpBig * (kMaxKpBig + 1) / 2];
  __shared__ __attribute__((aligned(16))) float sV[KB2];  // also eight rows of Gm (doubles) as scratch
  __shared__ double sH[kMaxKpBig], sHi[kMaxKpBig], sEig[kMaxKpBig];
  __shared__ double sT[5][kMaxKpBig];  // the tridiagonal eigensolver's vectors
  __shared__ int sOrd[kMaxKpBig];
  __shared__ __attribute__((aligned(16))) double cs[kMaxKpBig];
  __shared__ __attribute__((aligned(16))) int pairs[kMaxKpBig];
  __shared__ double red[kRedLen];
  const int64_t mi = blockIdx.x;
  const int tid = threadIdx.x;
  const int K = (int)kp;
  const int n = K + (K & 1);
  double* Gm = big + mi * 2 * KB2;
  double* T = Gm + KB2;
  float* Vs = (float*)(big + nm * 2 * KB2) + mi * KB2;
  const double* GmP = Gpart + (mi * 2) * nsplit * kp * kp;
  const double* GbP = Gpart + (mi * 2 + 1) * nsplit * kp * kp;
  // 1. Gb into sA (packed), Gm into the workspace, each summed over the row ranges in order
  for (int e = tid; e < n * n; e += kTC) {
    const int i = e / n, j = e % n;
    double gb = 0.0, gm = 0.0;
    if (i < K && j < K)
      for (int z = 0; z < nsplit; ++z) {
        gb += GbP[z * kp * kp + i * kp + j];
        gm += GmP[z * kp * kp + i * kp + j];
      }
    Gm[i * n + j] = gm;
    if (i <= j) sA[pk(i, j, n)] = gb;
  }
  __threadfence();
  __syncthreads();
  // 2. Gb = U^T U in place in sA (packed upper triangle), one barrier per row: step j updates
  // the trailing rows from the unscaled row j, A[i][k] -= A[j][i] A[j][k] / A[j][j]
  // (thread (ty, tx) of a 32 x 32 grid takes i in {ty + 32 a}, k in {tx + 32 b}), while row
  // j - 1, no longer read, is scaled into U; a pivot at or below 1e-10 of the largest
  // diagonal entry sends the core to the eigendecomposition of Gb instead (R close to rank
  // deficient), as in the core for kp <= 64
  bool chol = true;
  {
    const int ty = tid >> 5, tx = tid & 31;
    double mx = 0.0;
    for (int j = 0; j < K; ++j) mx = fmax(mx, sA[pk(j, j, n)]);
    const double thr = 1e-10 * mx;
    for (int j = 0; j < K; ++j) {
      const double piv = sA[pk(j, j, n)];
      if (j > 0) {
        const double inv = rsq64(sA[pk(j - 1, j - 1, n)]);
        for (int k = j + tid; k < K; k += kTC) sA[pk(j - 1, k, n)] *= inv;
      }
      if (!(piv > thr)) {  // uniform: every thread reads the same pivot
        chol = false;
        break;
      }
      const double rp = rcp64(piv);
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        const int i = ty + 32 * a;
        if (i <= j || i >= K) continue;
        const double aji = sA[pk(j, i, n)] * rp;
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          const int k = tx + 32 * b;
          if (k < i || k >= K) continue;
          sA[pk(i, k, n)] -= aji * sA[pk(j, k, n)];
        }
      }
      __syncthreads();
    }
    if (chol)
      for (int i = tid; i < K; i += kTC) sA[pk(i, i, n)] = sqrt(sA[pk(i, i, n)]);
  }
  __syncthreads();
  if (chol) {
    // 3. L = U^T (dense, lower) into T; T2 = Gm L over Gm, eight rows of Gm at a time
    // through LDS; P^T P = L^T T2 (upper triangle, packed) into sA
    for (int e = tid; e < n * n; e += kTC) {
      const int x = e / n, j = e % n;
      T[e] = (j <= x && x < K) ? sA[pk(j, x, n)] : 0.0;
    }
    __threadfence();
    __syncthreads();
    double* scr = reinterpret_cast<double*>(sV);
    for (int x0 = 0; x0 < K; x0 += 8) {
      for (int e = tid; e < 8 * n; e += kTC) {
        const int r = e / n, y = e % n;
        scr[e] = x0 + r < K ? Gm[(x0 + r) * n + y] : 0.0;
      }
      __syncthreads();
      {
        const int r = tid >> 7, j = tid & 127;
        if (x0 + r < K && j < K) {
          double sum = 0.0;
          for (int y = j; y < K; ++y) sum += scr[r * n + y] * T[y * n + j];
          Gm[(x0 + r) * n + j] = sum;
        }
      }
      __syncthreads();
    }
    __threadfence();
    __syncthreads();
    for (int e = tid; e < n * n; e += kTC) {
      const int i = e / n, j = e % n;
      if (i > j) continue;
      double sum = 0.0;
      if (j < K)
        for (int x = i; x < K; ++x) sum += T[x * n + i] * Gm[x * n + j];
      sA[pk(i, j, n)] = sum;
    }
    __syncthreads();
  } else {
    // 2'. Gb again, then Gb = Vb diag(lb) Vb^T by Jacobi; H = Vb diag(sqrt(lb)) over the kept
    // directions
    for (int e = tid; e < n * n; e += kTC) {
      const int i = e / n, j = e % n;
      if (i > j) continue;
      double gb = 0.0;
      if (j < K)
        for (int z = 0; z < nsplit; ++z) gb += GbP[z * kp * kp + i * kp + j];
      sA[pk(i, j, n)] = gb;
    }
    __syncthreads();
    jacobi_packed(sA, sV, n, cs, pairs, red);
    __syncthreads();
    if (tid == 0) {
      double lmax = 0.0;
      for (int j = 0; j < K; ++j) lmax = fmax(lmax, sA[pk(j, j, n)]);
      red[kRedMax] = lmax;
    }
    __syncthreads();
    for (int j = tid; j < n; j += kTC) {
      const double lb = j < K ? sA[pk(j, j, n)] : 0.0;
      const bool keep = lb > 1e-14 * red[kRedMax] && lb > 0.0;
      sH[j] = keep ? sqrt(lb) : 0.0;
      sHi[j] = keep ? 1.0 / sqrt(lb) : 0.0;
    }
    // keep Vb; T = Gm Vb; P^T P = H Vb^T T H into sA
    for (int e = tid; e < n * n; e += kTC) Vs[e] = sV[e];
    for (int e = tid; e < n * n; e += kTC) {
      const int i = e / n, j = e % n;
      double s = 0.0;
      for (int c = 0; c < n; ++c) s += Gm[i * n + c] * (double)sV[c * n + j];
      T[i * n + j] = s;
    }
    __threadfence();
    __syncthreads();
    for (int e = tid; e < n * n; e += kTC) {
      const int i = e / n, j = e % n;
      if (i > j) continue;
      double s = 0.0;
      for (int c = 0; c < n; ++c) s += (double)sV[c * n + i] * T[c * n + j];
      sA[pk(i, j, n)] = s * sH[i] * sH[j];
    }
    __syncthreads();
  }
  // sV = Vp: the leading r_a eigenpairs from the tridiagonal path on sA in place (a copy of
  // P^T P over Gm, no longer needed, for its check), or every pair by Jacobi when the check
  // fails
  const int np = n * (n + 1) / 2;
  for (int e = tid; e < np; e += kTC) Gm[e] = sA[e];
  __threadfence();
  __syncthreads();
  const int ra = (int)(r_a < kp ? r_a : kp);
  int live = ra;  // kept directions with weight (the others are completed by k_trunc_complete)
  if (eig_top<kMaxKpBig, true, float>(Gm, n, K, ra, sA, sV, reinterpret_cast<double*>(sV), sT[0], sT[1], sT[2],
                                      sT[3], sT[4], sEig, red)) {
    live = (int)red[kRedLive];
    for (int j = tid; j < K; j += kTC) sOrd[j] = j;
  } else {
    for (int e = tid; e < np; e += kTC) sA[e] = Gm[e];
    __syncthreads();
    jacobi_packed(sA, sV, n, cs, pairs, red);  // sV = Vp
    __syncthreads();
    if (tid == 0) {
      for (int j = 0; j < K; ++j) { sEig[j] = sA[pk(j, j, n)]; sOrd[j] = j; }
      for (int i = 1; i < K; ++i) {
        const int key = sOrd[i];
        int j = i - 1;
        while (j >= 0 && sEig[sOrd[j]] < sEig[key]) { sOrd[j + 1] = sOrd[j]; --j; }
        sOrd[j + 1] = key;
      }
    }
  }
  __syncthreads();
  const double s1 = sqrt(fmax(sEig[sOrd[0]], 0.0));
  for (int j = tid; j < K; j += kTC) sigma_out[mi * sigma_bstride + j] = (float)sqrt(fmax(sEig[sOrd[j]], 0.0));
  if (tid == 0) {  // directions 0 .. live - 1 carry weight; k_trunc_complete fills the rows past them
    int lv = 0;
    while (lv < live && lv < (int)r_a) {
      const double sa = sqrt(fmax(sEig[sOrd[lv]], 0.0));
      if (!(sa > 1e-30 * s1 && sa > 0.0)) break;
      ++lv;
    }
    live_out[mi] = lv;
  }
  // 3. Ca[a][c] = (Vb H Vp)[c][ord a] / s_a ;  Cb[c][a] = (Vb H^{-1} Vp)[c][ord a] * s_a
  double* Ca = Ca_all + mi * r_a * kp;
  double* Cb = Cb_all + mi * kp * r_a;
  if (chol) {  // Z = L^{-T} Vp for the kept columns (over Gm): 16 lanes per column,
               // entries x = t + 16 q of the column in registers, the substitution upwards
    const int a = tid >> 4, t = tid & 15;
    if (a < (int)r_a) {
      const int col = sOrd[a];
      double zq[8] = {0.0, 0.0, 0.0, 0.0, 0.0, 0.0, 0.0, 0.0};
      for (int c = K - 1; c >= 0; --c) {
        double sum = 0.0;
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          const int x = t + 16 * q;
          if (x > c && x < K) sum += T[x * n + c] * zq[q];
        }
        sum = seg16_sum(sum);
        const double zc = ((double)sV[c * n + col] - sum) / T[c * n + c];
#pragma unroll
        for (int q = 0; q < 8; ++q)
          if (c == t + 16 * q) zq[q] = zc;
      }
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const int x = t + 16 * q;
        if (x < K) Gm[x * n + col] = zq[q];
      }
    }
    __threadfence();
    __syncthreads();
  }
  for (int e = tid; e < (int)(r_a * kp); e += kTC) {
    const int a = e % (int)r_a, c = e / (int)r_a;  // lanes along a
    const int col = sOrd[a];
    const double sa = sqrt(fmax(sEig[col], 0.0));
    double u = 0.0, v = 0.0;
    if (chol) {  // Ca from L Vp, Cb from Z
      for (int x = 0; x <= c; ++x) u += T[c * n + x] * (double)sV[x * n + col];
      v = Gm[c * n + col];
    } else {
      for (int x = 0; x < n; ++x) {
        const double vb = (double)Vs[c * n + x], vp = (double)sV[x * n + col];
        u += vb * sH[x] * vp;
        v += vb * sHi[x] * vp;
      }
    }
    const bool on = a < live && sa > 1e-30 * s1 && sa > 0.0;
    Ca[a * kp + c] = on ? u / sa : 0.0;
    Cb[c * r_a + a] = on ? v * sa : 0.0;
  }
}

// a_out[a][i] = sum_c Ca[a][c] M[i][c];  b_out[i][a] = sum_c R[c][i] Cb[c][a]  for kp <= 128,
// r_a <= 64: 64 rows i per workgroup, kp in chunks of 32 through LDS; thread t owns row
// t % 64 and the ranks a = t / 64 + 4u (fp64 sums in the order of c).
__global__ __launch_bounds__(kT) void k_trunc_apply_tiled(int64_t d, int64_t kp, int64_t r_a,
                                                          const float* __restrict__ M, int64_t m_bstride,
                                                          const float* __restrict__ R, int64_t r_bstride,
                                                          int64_t r_group, const double* __restrict__ Ca_all,
                                                          const double* __restrict__ Cb_all, float* __restrict__ a_out,
                                                          int64_t a_bstride, float* __restrict__ b_out,
                                                          int64_t b_bstride) {
  __shared__ float sM[64][33];
  __shared__ float sR[32][65];
  __shared__ double sCa[64][33];
  __shared__ double sCb[32][65];
  const int64_t mi = blockIdx.y;
  const int64_t i0 = (int64_t)blockIdx.x * 64;
  const int tid = threadIdx.x, r = tid & 63, q = tid >> 6;
  const float* Mm = M + mi * m_bstride;
  const float* Rm = R + (mi / r_group) * r_bstride;
  const double* Ca = Ca_all + mi * r_a * kp;
  const double* Cb = Cb_all + mi * kp * r_a;
  double sa[16], sb[16];
#pragma unroll
  for (int u = 0; u < 16; ++u) { sa[u] = 0.0; sb[u] = 0.0; }
  for (int64_t c0 = 0; c0 < kp; c0 += 32) {
    __syncthreads();
    for (int e = tid; e < 64 * 32; e += kT) {
      const int rr = e / 32, cc = e % 32;
      sM[rr][cc] = (i0 + rr < d && c0 + cc < kp) ? Mm[(i0 + rr) * kp + c0 + cc] : 0.f;
      const int cr = e / 64, ir = e % 64;
      sR[cr][ir] = (i0 + ir < d && c0 + cr < kp) ? Rm[(c0 + cr) * d + i0 + ir] : 0.f;
      sCa[rr][cc] = (rr < r_a && c0 + cc < kp) ? Ca[rr * kp + c0 + cc] : 0.0;
      sCb[cr][ir] = (ir < r_a && c0 + cr < kp) ? Cb[(c0 + cr) * r_a + ir] : 0.0;
    }
    __syncthreads();
    for (int cc = 0; cc < 32; ++cc) {
      const double mv = (double)sM[r][cc], rv = (double)sR[cc][r];
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        const int a = q + 4 * u;
        sa[u] += sCa[a][cc] * mv;
        sb[u] += rv * sCb[cc][a];
      }
    }
  }
  const int64_t i = i0 + r;
  if (i < d)
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      const int a = q + 4 * u;
      if (a < r_a) {
        a_out[mi * a_bstride + a * d + i] = (float)sa[u];
        b_out[mi * b_bstride + i * r_a + a] = (float)sb[u];
      }
    }
}

// One workgroup per matrix: the small factors Ca, Cb (kp <= 64).  First Gb = L L^T by
// Cholesky (fp64, in LDS): when every pivot exceeds 1e-10 of the largest diagonal entry,
// any square root of Gb serves for H (W = (M L)(L^{-1} R), the second factor with
// orthonormal rows), so one eigensolve remains, of P^T P = L^T Gm L = Vp diag(s^2) Vp^T, and
//   Ca[a][c] = (L Vp)[c][a] / s_a,   Cb[c][a] = (L^{-T} Vp)[c][a] s_a.
// Otherwise (R close to rank deficient) Gb = Vb diag(lb) Vb^T by Jacobi, directions with
// lb <= 1e-14 max lb dropped, and H = Vb diag(sqrt(lb)) as in the file comment.  The
// symmetric matrices of the eigensolves are packed in LDS (jacobi_packed); Gm, the factor of
// Gb and the eigenvectors (fp64) stay in LDS.
__global__ __launch_bounds__(kTC) void k_trunc_core(int64_t kp, int64_t r_a, const double* __restrict__ Gpart,
                                                    int nsplit, double* __restrict__ Ca_all,
                                                    double* __restrict__ Cb_all, float* __restrict__ sigma_out,
                                                    int64_t sigma_bstride, int32_t* __restrict__ live_out) {
  constexpr int KB2 = kMaxKp * kMaxKp;
  __shared__ double sA[kMaxKp * (kMaxKp + 1) / 2];
  __shared__ double sV[KB2];   // eigenvectors of the current eigensolve; T = Gm H in between
  __shared__ double sVb[KB2];  // Gb, then its factor: L (Cholesky) or Vb (Jacobi)
  __shared__ double sG[KB2];   // Gm; L^{-T} Vp after the eigensolve (Cholesky path)
  __shared__ double sH[kMaxKp], sHi[kMaxKp], sEig[kMaxKp];
  __shared__ double sT[5][kMaxKp];  // the tridiagonal eigensolver's vectors
  __shared__ int sOrd[kMaxKp];
  __shared__ __attribute__((aligned(16))) double cs[kMaxKp];
  __shared__ __attribute__((aligned(16))) int pairs[kMaxKp];
  __shared__ double red[kRedLen];
  const int64_t mi = blockIdx.x;
  const int tid = threadIdx.x;
  const int K = (int)kp;
  const int n = K + (K & 1);  // even size for the tournament ordering
  const double* GmP = Gpart + (mi * 2) * nsplit * kp * kp;
  const double* GbP = Gpart + (mi * 2 + 1) * nsplit * kp * kp;
  // 1. Gm into sG and Gb into sVb (n x n, zero padded), each summed over the row ranges in order
  for (int e = tid; e < n * n; e += kTC) {
    const int i = e / n, j = e % n;
    double gb = 0.0, gm = 0.0;
    if (i < K && j < K)
      for (int z = 0; z < nsplit; ++z) {
        gb += GbP[z * kp * kp + i * kp + j];
        gm += GmP[z * kp * kp + i * kp + j];
      }
    sG[e] = gm;
    sVb[e] = gb;
  }
  __syncthreads();
  // 2. Gb = L L^T (L in the lower triangle of sVb), or a failed pivot.  One barrier per
  // step: step j updates the trailing lower triangle from the unscaled column j,
  // A[i][c] -= A[i][j] A[c][j] / A[j][j] (thread (ty, tx) of a 32 x 32 grid takes i in
  // {ty, ty + 32}, c in {tx, tx + 32}), while column j - 1, no longer read, is scaled into L.
  {
    const int ty = tid >> 5, tx = tid & 31;
    double mx = 0.0;
    for (int j = 0; j < K; ++j) mx = fmax(mx, sVb[j * n + j]);
    const double thr = 1e-10 * mx;
    bool fail = false;
    int j = 0;
    for (; j < K; ++j) {
      const double piv = sVb[j * n + j];
      if (j > 0) {  // column j - 1 into L
        const double pj = sVb[(j - 1) * n + j - 1];  // its pivot, still unscaled
        const double inv = rsq64(pj);
        for (int i = j + tid; i < K; i += kTC) sVb[i * n + j - 1] *= inv;
      }
      if (!(piv > thr)) {  // uniform: every thread reads the same pivot
        fail = true;
        break;
      }
      const double rp = rcp64(piv);
#pragma unroll
      for (int a = 0; a < 2; ++a) {
        const int i = ty + 32 * a;
        if (i <= j || i >= K) continue;
        const double aij = sVb[i * n + j] * rp;
#pragma unroll
        for (int b = 0; b < 2; ++b) {
          const int c = tx + 32 * b;
          if (c <= j || c > i) continue;
          sVb[i * n + c] -= aij * sVb[c * n + j];
        }
      }
      __syncthreads();
    }
    if (!fail)  // the diagonal of L (the last column has nothing below it)
      for (int i = tid; i < K; i += kTC) sVb[i * n + i] = sqrt(sVb[i * n + i]);
    if (tid == 0) red[kRedFail] = fail ? 1.0 : 0.0;
  }
  __syncthreads();
  const bool chol = red[kRedFail] == 0.0;
  if (chol) {
    // 3. T = Gm L (into sV), P^T P = L^T T (upper triangle, packed; zero padding)
    for (int e = tid; e < K * K; e += kTC) {
      const int i = e / K, c = e % K;
      double s = 0.0;
      for (int x = c; x < K; ++x) s += sG[i * n + x] * sVb[x * n + c];
      sV[i * n + c] = s;
    }
    __syncthreads();
    for (int e = tid; e < n * n; e += kTC) {
      const int i = e / n, j = e % n;
      if (i > j) continue;
      double s = 0.0;
      if (j < K)
        for (int x = i; x < K; ++x) s += sVb[x * n + i] * sV[x * n + j];
      sA[pk(i, j, n)] = s;
    }
    __syncthreads();
  } else {
    // 3'. Gb = Vb diag(lb) Vb^T; H = Vb diag(sqrt(lb)) over the kept directions: those above
    // 1e-12 ||Gb|| from the tridiagonal path (the others get no vector, lb = 0), or every
    // pair by Jacobi (kept above 1e-14 of the largest) when its check fails
    for (int e = tid; e < n * n; e += kTC) {
      const int i = e / n, j = e % n;
      if (i > j) continue;
      double gb = 0.0;
      if (j < K)
        for (int z = 0; z < nsplit; ++z) gb += GbP[z * kp * kp + i * kp + j];
      sA[pk(i, j, n)] = gb;
    }
    __syncthreads();
    if (eig_top<kMaxKp, false, double>(sA, n, K, K, sV, sV, sVb, sT[0], sT[1], sT[2], sT[3], sT[4], sEig, red)) {
      const int nb = (int)red[kRedLive];
      for (int j = tid; j < n; j += kTC) {
        const double lb = j < nb ? sEig[j] : 0.0;
        const bool keep = lb > 0.0;
        sH[j] = keep ? sqrt(lb) : 0.0;
        sHi[j] = keep ? 1.0 / sqrt(lb) : 0.0;
      }
    } else {
      jacobi_packed<double>(sA, sV, n, cs, pairs, red);
      __syncthreads();
      if (tid == 0) {
        double lmax = 0.0;
        for (int j = 0; j < K; ++j) lmax = fmax(lmax, sA[pk(j, j, n)]);
        red[kRedMax] = lmax;
      }
      __syncthreads();
      for (int j = tid; j < n; j += kTC) {
        const double lb = j < K ? sA[pk(j, j, n)] : 0.0;
        const bool keep = lb > 1e-14 * red[kRedMax] && lb > 0.0;
        sH[j] = keep ? sqrt(lb) : 0.0;
        sHi[j] = keep ? 1.0 / sqrt(lb) : 0.0;
      }
    }
    __syncthreads();
    for (int e = tid; e < n * n; e += kTC) sVb[e] = sV[e];
    __syncthreads();
    // T = Gm Vb (into sV), then P^T P = H Vb^T T H (upper triangle, packed)
    for (int e = tid; e < n * n; e += kTC) {
      const int i = e / n, j = e % n;
      double s = 0.0;
      for (int c = 0; c < n; ++c) s += sG[i * n + c] * sVb[c * n + j];
      sV[e] = s;
    }
    __syncthreads();
    for (int e = tid; e < n * n; e += kTC) {
      const int i = e / n, j = e % n;
      if (i > j) continue;
      double s = 0.0;
      for (int c = 0; c < n; ++c) s += sVb[c * n + i] * sV[c * n + j];
      sA[pk(i, j, n)] = s * sH[i] * sH[j];
    }
    __syncthreads();
  }
  // sV = Vp: the leading r_a eigenpairs from the tridiagonal path, or every pair by Jacobi
  // when its check fails
  const int ra = (int)(r_a < kp ? r_a : kp);
  int live = ra;  // kept directions with weight (the others are completed by k_trunc_complete)
  if (eig_top<kMaxKp, false, double>(sA, n, K, ra, sV, sV, sG, sT[0], sT[1], sT[2], sT[3], sT[4], sEig, red)) {
    live = (int)red[kRedLive];
    for (int j = tid; j < K; j += kTC) sOrd[j] = j;
  } else {
    jacobi_packed<double>(sA, sV, n, cs, pairs, red);
    __syncthreads();
    if (tid == 0) {
      // order by decreasing eigenvalue (insertion sort on indices)
      for (int j = 0; j < K; ++j) { sEig[j] = sA[pk(j, j, n)]; sOrd[j] = j; }
      for (int i = 1; i < K; ++i) {
        const int key = sOrd[i];
        int j = i - 1;
        while (j >= 0 && sEig[sOrd[j]] < sEig[key]) { sOrd[j + 1] = sOrd[j]; --j; }
        sOrd[j + 1] = key;
      }
    }
  }
  __syncthreads();
  if (chol) {  // Z = L^{-T} Vp for the kept columns (into sG): 16 lanes per column, entries
               // x = t + 16 q of the column in registers while the substitution runs upwards
    const int a = tid >> 4, t = tid & 15;
    if (a < ra) {
      const int col = sOrd[a];
      double zq[4] = {0.0, 0.0, 0.0, 0.0};
      for (int c = K - 1; c >= 0; --c) {
        double sum = 0.0;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int x = t + 16 * q;
          if (x > c && x < K) sum += sVb[x * n + c] * zq[q];
        }
        sum = seg16_sum(sum);
        const double zc = (sV[c * n + col] - sum) / sVb[c * n + c];
#pragma unroll
        for (int q = 0; q < 4; ++q)
          if (c == t + 16 * q) zq[q] = zc;
      }
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int x = t + 16 * q;
        if (x < K) sG[x * n + col] = zq[q];
      }
    }
  }
  __syncthreads();
  const double s1 = sqrt(fmax(sEig[sOrd[0]], 0.0));
  for (int j = tid; j < K; j += kTC) sigma_out[mi * sigma_bstride + j] = (float)sqrt(fmax(sEig[sOrd[j]], 0.0));
  if (tid == 0) {  // directions 0 .. live - 1 carry weight; k_trunc_complete fills the rows past them
    int lv = 0;
    while (lv < live && lv < (int)r_a) {
      const double sa = sqrt(fmax(sEig[sOrd[lv]], 0.0));
      if (!(sa > 1e-30 * s1 && sa > 0.0)) break;
      ++lv;
    }
    live_out[mi] = lv;
  }
  // 4. Ca[a][c] = (H Vp)[c][ord a] / s_a ;  Cb[c][a] = (H^{-T} Vp)[c][ord a] * s_a
  double* Ca = Ca_all + mi * r_a * kp;
  double* Cb = Cb_all + mi * kp * r_a;
  for (int e = tid; e < (int)(r_a * kp); e += kTC) {
    const int a = e % (int)r_a, c = e / (int)r_a;  // lanes along a: rows of sVb read once per wave
    const int col = sOrd[a];
    const double sa = sqrt(fmax(sEig[col], 0.0));
    double u = 0.0, v = 0.0;
    if (chol) {
      for (int x = 0; x <= c; ++x) u += sVb[c * n + x] * sV[x * n + col];
      v = sG[c * n + col];
    } else {
      for (int x = 0; x < n; ++x) {
        const double vb = sVb[c * n + x], vp = sV[x * n + col];
        u += vb * sH[x] * vp;
        v += vb * sHi[x] * vp;
      }
    }
    const bool on = a < live && sa > 1e-30 * s1 && sa > 0.0;
    Ca[a * kp + c] = on ? u / sa : 0.0;
    Cb[c * r_a + a] = on ? v * sa : 0.0;
  }
}

// a_out[a][i] = sum_c Ca[a][c] M[i][c];  b_out[i][a] = sum_c R[c][i] Cb[c][a]  (kp <= 64): one
// thread per row i and kRA ranks a0 = kRA blockIdx.z .. (fp64 sums in the order of c), the
// small factors in LDS ([c][a], read by every lane at once), M read by rows as float4 when
// aligned, the rows of b_out written as float4 when r_a % 4 == 0.
constexpr int kRA = 16;
__global__ __launch_bounds__(kT) void k_trunc_apply(int64_t d, int64_t kp, int64_t r_a, const float* __restrict__ M,
                                                    int64_t m_bstride, const float* __restrict__ R, int64_t r_bstride,
                                                    int64_t r_group, const double* __restrict__ Ca_all,
                                                    const double* __restrict__ Cb_all, float* __restrict__ a_out,
                                                    int64_t a_bstride, float* __restrict__ b_out, int64_t b_bstride) {
  __shared__ __attribute__((aligned(16))) double sCa[kMaxKp * kRA];  // [c][a - a0]
  __shared__ __attribute__((aligned(16))) double sCb[kMaxKp * kRA];  // [c][a - a0]
  const int64_t mi = blockIdx.y;
  const int a0 = kRA * (int)blockIdx.z;
  for (int e = threadIdx.x; e < (int)kp * kRA; e += kT) {
    const int c = e / kRA, u = e % kRA, a = a0 + u;
    sCa[e] = a < r_a ? Ca_all[mi * r_a * kp + (int64_t)a * kp + c] : 0.0;
    sCb[e] = a < r_a ? Cb_all[mi * kp * r_a + (int64_t)c * r_a + a] : 0.0;
  }
  __syncthreads();
  const int64_t i = (int64_t)blockIdx.x * kT + threadIdx.x;
  if (i >= d) return;
  const float* Mi = M + mi * m_bstride + i * kp;
  const float* Rm = R + (mi / r_group) * r_bstride;
  const bool mv4 = (kp & 3) == 0 && (m_bstride & 3) == 0 && (((uintptr_t)M) & 15) == 0;
  double sa[kRA], sb[kRA];
#pragma unroll
  for (int u = 0; u < kRA; ++u) sa[u] = sb[u] = 0.0;
  for (int c0 = 0; c0 < kp; c0 += 4) {
    float mv[4], rv[4];
    if (mv4) {
      const float4 t = *(const float4*)(Mi + c0);
      mv[0] = t.x; mv[1] = t.y; mv[2] = t.z; mv[3] = t.w;
    } else {
#pragma unroll
      for (int t = 0; t < 4; ++t) mv[t] = c0 + t < kp ? Mi[c0 + t] : 0.f;
    }
#pragma unroll
    for (int t = 0; t < 4; ++t) rv[t] = c0 + t < kp ? Rm[(int64_t)(c0 + t) * d + i] : 0.f;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      if (c0 + t >= kp) break;
      const double* ca = sCa + (c0 + t) * kRA;
      const double* cb = sCb + (c0 + t) * kRA;
#pragma unroll
      for (int u = 0; u < kRA; ++u) {
        sa[u] += ca[u] * (double)mv[t];
        sb[u] += (double)rv[t] * cb[u];
      }
    }
  }
  const int na = (int)(r_a - a0 < kRA ? r_a - a0 : kRA);
#pragma unroll
  for (int u = 0; u < kRA; ++u)
    if (u < na) a_out[mi * a_bstride + (int64_t)(a0 + u) * d + i] = (float)sa[u];
  float* bo = b_out + mi * b_bstride + i * r_a + a0;
  if ((r_a & 3) == 0 && (b_bstride & 3) == 0 && (((uintptr_t)b_out) & 15) == 0) {
#pragma unroll
    for (int u = 0; u < kRA; u += 4)
      if (u < na) *(float4*)(bo + u) = make_float4((float)sb[u], (float)sb[u + 1], (float)sb[u + 2], (float)sb[u + 3]);
  } else {
#pragma unroll
    for (int u = 0; u < kRA; ++u)
      if (u < na) bo[u] = (float)sb[u];
  }
}

// out[i][j] = sum_c L(i, c) R(c, j) with general strides (fp64 accumulation).
__global__ void k_lowrank_product(int64_t rows, int64_t cols, int64_t kk, const float* __restrict__ L,
                                  int64_t l_bstride, int64_t l_si, int64_t l_sc, const float* __restrict__ R,
                                  int64_t r_bstride, int64_t r_group, int64_t r_sc, int64_t r_sj,
                                  float* __restrict__ out, int64_t out_bstride) {
  const int64_t mi = blockIdx.z;
  const int64_t i = blockIdx.y;
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= cols) return;
  const float* Lm = L + mi * l_bstride + i * l_si;
  const float* Rm = R + (mi / r_group) * r_bstride + j * r_sj;
  double s = 0.0;
  for (int64_t c = 0; c < kk; ++c) s += (double)Lm[c * l_sc] * (double)Rm[c * r_sc];
  out[mi * out_bstride + i * cols + j] = (float)s;
}

__global__ void k_fill_zero(int32_t* p, int64_t cnt) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < cnt) p[i] = 0;
}

// Rows rho = live[mi] .. r_a - 1 of a_out (matrix mi), whose directions carry no weight
// (their b_out columns are zero), completed to orthonormal rows orthogonal to the rho live
// rows L: columns rho .. r_a - 1 of the orthogonal H = I - Y T Y^T whose first rho columns are
// L^T up to signs, H built from L by Householder reconstruction (Ballard et al., 2014): the
// LU factorization without pivoting of the top rho x rho block of L^T minus diag(s), each
// sign s_k opposite to the pivot it is subtracted from, gives Y's top block Y1 (unit lower)
// and U; Y's other rows are L[:, i]^T U^{-1}, and T = -U diag(s) Y1^{-T}.  With
// t_j = T Y[rho + j, :]^T and w_j = U^{-1} t_j the rows are
//   X[j][i] = [i = rho + j] - sum_q w_j[q] L[q][i] + [i < rho] s_i w_j[i].
// Workgroup (mi, y) writes coordinates [y kCSpan, (y + 1) kCSpan) of the rows of matrix mi
// (the matrices without such rows return at once): the small factors in LDS (fp64, each
// workgroup of a matrix alike), then per coordinate i a thread takes L[:, i] 16 rows at a
// time in registers (w zero-padded to a multiple of 16) and writes the r_a - rho rows.
constexpr int kTCC = 256;
constexpr int kCSpan = 1024;
__global__ __launch_bounds__(kTCC) void k_trunc_complete(int64_t d, int64_t r_a, const int32_t* __restrict__ live,
                                                         float* __restrict__ a_out, int64_t a_bstride) {
  constexpr int LD = kMaxRank + 1;
  __shared__ double sA[kMaxRank][LD];   // L^T top block - diag(s): LU in place; later Y rows, then w
  __shared__ double sUi[kMaxRank][LD];  // U^{-1}
  __shared__ double sZ[kMaxRank][LD];   // Y1^{-1}; later t
  __shared__ double sT[kMaxRank][LD];   // T
  __shared__ double sSg[kMaxRank];
  const int64_t mi = blockIdx.x;
  const int rho = live[mi];
  const int D = (int)r_a - rho;
  if (D <= 0) return;
  float* L = a_out + mi * a_bstride;
  const int tid = threadIdx.x;
  for (int e = tid; e < rho * rho; e += kTCC) sA[e / rho][e % rho] = (double)L[(int64_t)(e % rho) * d + e / rho];
  __syncthreads();
  for (int k = 0; k < rho; ++k) {
    if (tid == 0) {
      const double sg = sA[k][k] >= 0.0 ? -1.0 : 1.0;
      sSg[k] = sg;
      sA[k][k] -= sg;
    }
    __syncthreads();
    for (int i = k + 1 + tid; i < rho; i += kTCC) sA[i][k] /= sA[k][k];
    __syncthreads();
    const int rem = rho - k - 1;
    for (int e = tid; e < rem * rem; e += kTCC) {
      const int i = k + 1 + e / rem, c = k + 1 + e % rem;
      sA[i][c] -= sA[i][k] * sA[k][c];
    }
    __syncthreads();
  }
  if (tid < rho) {  // column tid of U^{-1}
    const int c = tid;
    for (int i = rho - 1; i >= 0; --i) {
      double x = 0.0;
      if (i <= c) {
        x = i == c ? 1.0 : 0.0;
        for (int k = i + 1; k <= c; ++k) x -= sA[i][k] * sUi[k][c];
        x /= sA[i][i];
      }
      sUi[i][c] = x;
    }
  } else if (tid >= 64 && tid < 64 + rho) {  // column c of Y1^{-1}
    const int c = tid - 64;
    for (int i = 0; i < rho; ++i) {
      double z = i == c ? 1.0 : 0.0;
      if (i > c)
        for (int k = c; k < i; ++k) z -= sA[i][k] * sZ[k][c];
      sZ[i][c] = z;
    }
  }
  __syncthreads();
  for (int e = tid; e < rho * rho; e += kTCC) {  // T = -U diag(s) Y1^{-T}
    const int a = e / rho, b = e % rho;
    double t = 0.0;
    for (int k = a; k <= b; ++k) t -= sA[a][k] * sSg[k] * sZ[b][k];
    sT[a][b] = t;
  }
  __syncthreads();
  for (int e = tid; e < D * rho; e += kTCC) {  // Y[rho + j][p] = sum_q L[q][rho + j] U^{-1}[q][p]
    const int j = e / rho, p = e % rho;
    double y = 0.0;
    for (int q = 0; q <= p; ++q) y += (double)L[(int64_t)q * d + rho + j] * sUi[q][p];
    sA[j][p] = y;
  }
  __syncthreads();
  for (int e = tid; e < D * rho; e += kTCC) {  // t_j = T Y[rho + j]^T
    const int j = e / rho, a = e % rho;
    double t = 0.0;
    for (int b = a; b < rho; ++b) t += sT[a][b] * sA[j][b];
    sZ[j][a] = t;
  }
  __syncthreads();
  const int rho16 = rho > 0 ? (rho + 15) & ~15 : 16;
  for (int e = tid; e < D * rho16; e += kTCC) {  // w_j = U^{-1} t_j, zero past rho
    const int j = e / rho16, q = e % rho16;
    double w = 0.0;
    for (int a = q; a < rho; ++a) w += sUi[q][a] * sZ[j][a];
    sA[j][q] = w;
  }
  __syncthreads();
  const int64_t i_end = (int64_t)(blockIdx.y + 1) * kCSpan < d ? (int64_t)(blockIdx.y + 1) * kCSpan : d;
  for (int64_t i = (int64_t)blockIdx.y * kCSpan + tid; i < i_end; i += kTCC) {
    for (int q0 = 0; q0 == 0 || q0 < rho; q0 += 16) {  // once when rho = 0
      double l[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) l[u] = q0 + u < rho ? (double)L[(int64_t)(q0 + u) * d + i] : 0.0;
      for (int j = 0; j < D; ++j) {
        float* out = L + (int64_t)(rho + j) * d + i;
        double x;
        if (q0 == 0) {
          x = i == rho + j ? 1.0 : 0.0;
          if (i < rho) x += sSg[i] * sA[j][i];
        } else {
          x = (double)*out;
        }
#pragma unroll
        for (int u = 0; u < 16; ++u) x -= sA[j][q0 + u] * l[u];
        *out = (float)x;
      }
    }
  }
}

}  // namespace

hipError_t launch_lowrank_product(hipStream_t s, int64_t nmat, int64_t rows, int64_t cols, int64_t kk,
                                  const float* L, int64_t l_bstride, int64_t l_ld, const float* R,
                                  int64_t r_bstride, int64_t r_group, int64_t r_ld, float* out,
                                  int64_t out_bstride) {
  dim3 grid((unsigned)((cols + 255) / 256), (unsigned)rows, (unsigned)nmat);
  k_lowrank_product<<<grid, 256, 0, s>>>(rows, cols, kk, L, l_bstride, l_ld, 1, R, r_bstride, r_group, r_ld, 1, out,
                                         out_bstride);
  return hipGetLastError();
}

int trunc_splits(int64_t d) {
  const int64_t s = d / 256;
  return (int)(s < 1 ? 1 : (s > 16 ? 16 : s));
}

size_t lowrank_truncate_ws(int64_t nm, int64_t d, int64_t kp, int64_t r_a) {
  size_t s = align256(sizeof(double) * nm * 2 * trunc_splits(d) * kp * kp);
  s += 2 * align256(sizeof(double) * nm * kp * r_a);
  s += align256(sizeof(int32_t) * nm);  // directions with weight per matrix
  if (kp > kMaxKp)  // Gm, T (fp64) and the float copy of Vb per matrix
    s += align256(sizeof(double) * nm * 2 * kMaxKpBig * kMaxKpBig) + align256(sizeof(float) * nm * kMaxKpBig * kMaxKpBig);
  return s;
}

hipError_t launch_lowrank_truncate(const TruncArgs& a) {
  char* p = a.ws;
  const int ns = trunc_splits(a.d);
  double* Gpart = (double*)p; p += align256(sizeof(double) * a.nm * 2 * ns * a.kp * a.kp);
  double* Ca = (double*)p; p += align256(sizeof(double) * a.nm * a.kp * a.r_a);
  double* Cb = (double*)p; p += align256(sizeof(double) * a.nm * a.kp * a.r_a);
  int32_t* live = (int32_t*)p; p += align256(sizeof(int32_t) * a.nm);
  k_fill_zero<<<(unsigned)((a.nm + 255) / 256), 256, 0, a.stream>>>(a.dev_info, a.nm);
  if (a.kp <= kMaxKp) {
    k_small_grams<kMaxKp><<<dim3((unsigned)a.nm, 2, (unsigned)ns), kT, 0, a.stream>>>(
        a.d, a.kp, a.m, a.m_bstride, a.r, a.r_bstride, a.r_group, ns, Gpart);
    k_trunc_core<<<(unsigned)a.nm, kTC, 0, a.stream>>>(a.kp, a.r_a, Gpart, ns, Ca, Cb, a.sigma_out, a.sigma_bstride,
                                                       live);
    k_trunc_apply<<<dim3((unsigned)((a.d + kT - 1) / kT), (unsigned)a.nm, (unsigned)((a.r_a + kRA - 1) / kRA)), kT, 0,
                    a.stream>>>(
        a.d, a.kp, a.r_a, a.m, a.m_bstride, a.r, a.r_bstride, a.r_group, Ca, Cb, a.a_out, a.a_bstride, a.b_out,
        a.b_bstride);
  } else {
    double* big = (double*)p;
    k_small_grams<kMaxKpBig><<<dim3((unsigned)a.nm, 2, (unsigned)ns), kT, 0, a.stream>>>(
        a.d, a.kp, a.m, a.m_bstride, a.r, a.r_bstride, a.r_group, ns, Gpart);
    k_trunc_core_big<<<(unsigned)a.nm, kTC, 0, a.stream>>>(a.nm, a.kp, a.r_a, Gpart, ns, big, Ca, Cb, a.sigma_out,
                                                           a.sigma_bstride, live);
    k_trunc_apply_tiled<<<dim3((unsigned)((a.d + 63) / 64), (unsigned)a.nm), kT, 0, a.stream>>>(
        a.d, a.kp, a.r_a, a.m, a.m_bstride, a.r, a.r_bstride, a.r_group, Ca, Cb, a.a_out, a.a_bstride, a.b_out,
        a.b_bstride);
  }
  k_trunc_complete<<<dim3((unsigned)a.nm, (unsigned)((a.d + kCSpan - 1) / kCSpan)), kTCC, 0, a.stream>>>(
      a.d, a.r_a, live, a.a_out, a.a_bstride);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !a.w_dense_out) return e;
  // W_r[i][j] = sum_a a_out[a][i] b_out[j][a]
  dim3 grid((unsigned)((a.d + 255) / 256), (unsigned)a.d, (unsigned)a.nm);
  k_lowrank_product<<<grid, 256, 0, a.stream>>>(a.d, a.d, a.r_a, a.a_out, a.a_bstride, 1, a.d, a.b_out, a.b_bstride,
                                                1, 1, a.r_a, a.w_dense_out, a.w_bstride);
  return hipGetLastError();
}

// ------------------------------------------------------------------ projected form (Eqs. 6-9)

namespace {

// T1[b][i][a] = sum_j S_sym[i][j] PA[a][j]  (fp64, d x r_a); S_sym from the upper triangle.
template <typename ST>
__global__ void k_proj_sa(int64_t d, int64_t r_a, const ST* __restrict__ S, int64_t s_bstride,
                          const float* __restrict__ PA, int64_t pa_bstride, double* __restrict__ T1) {
  const int64_t b = blockIdx.y;
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= d * r_a) return;
  const int64_t i = e / r_a, a = e % r_a;
  const ST* Sb = S + b * s_bstride;
  const float* P = PA + b * pa_bstride + a * d;
  double s = 0.0;
  for (int64_t j = 0; j < i; ++j) s += (double)Sb[j * d + i] * (double)P[j];
  for (int64_t j = i; j < d; ++j) s += (double)Sb[i * d + j] * (double)P[j];
  T1[b * d * r_a + e] = s;
}

// The same product for fp32 S on the fp32 matrix cores (v_mfma_f32_32x32x2f32), reading S
// once per use with coalesced loads.  One workgroup per (64-row panel I, block b); the
// panel's rows of the symmetric S are staged 64 columns at a time: chunks right of the
// diagonal straight from the stored upper triangle, chunks left of it as the transposes of
// the stored tiles above the diagonal, the diagonal chunk mirrored in LDS; the chunk of
// PA^T beside it.  The next chunk's loads are issued before the current chunk's products
// (16-byte loads when d % 4 == 0).  Wave w forms the panel (64 x RA) over columns
// 16 w .. 16 w + 15 of every chunk, and the four partial panels are added in a fixed
// order: deterministic.
constexpr int kPS = 64;        // panel rows and chunk columns
constexpr int kPSL = kPS + 1;  // LDS row stride (odd: column reads spread over the banks)
template <int RA, bool V4>
__global__ __launch_bounds__(256) void k_proj_sa_mfma(int64_t d, int64_t r_a, const float* __restrict__ S,
                                                      int64_t s_bstride, const float* __restrict__ PA,
                                                      int64_t pa_bstride, double* __restrict__ T1) {
  constexpr int NCB = RA / 32;
  constexpr int SQ = kPS * kPS / 4 / 256;  // float4 groups of the S tile per thread
  constexpr int AQ = RA * kPS / 4 / 256;   // ... of the PA tile
  __shared__ float sS[kPS * kPSL];   // [row i][column j] of the panel chunk
  __shared__ float sA[RA * kPSL];    // [adapter row a][column j]
  __shared__ float sRed[4][kPS][RA + 1];
  const int64_t b = blockIdx.y;
  const int I = blockIdx.x;
  const int64_t i0 = (int64_t)I * kPS;
  const float* Sb = S + b * s_bstride;
  const float* Pb = PA + b * pa_bstride;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  f32x16_t acc[2][NCB];
#pragma unroll
  for (int rb = 0; rb < 2; ++rb)
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[rb][cb][r] = 0.f;
  const int nch = (int)((d + kPS - 1) / kPS);
  float4 vS[SQ], vA[AQ];
  // group e of a tile: row e / 16, columns 4 (e % 16) .. + 3
  auto load4 = [&](const float* base, int64_t row, int64_t col, int64_t rows_ok) {
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
    if (row < rows_ok) {
      if (V4) {
        if (col < d) v = *(const float4*)(base + row * d + col);
      } else {
        v.x = col < d ? base[row * d + col] : 0.f;
        v.y = col + 1 < d ? base[row * d + col + 1] : 0.f;
        v.z = col + 2 < d ? base[row * d + col + 2] : 0.f;
        v.w = col + 3 < d ? base[row * d + col + 3] : 0.f;
      }
    }
    return v;
  };
  auto load = [&](int J) {  // stored tile rows r0.., columns c0.. (transposed when left of the diagonal)
    const int64_t j0 = (int64_t)J * kPS;
    const bool left = J < I;
    const int64_t r0 = left ? j0 : i0, c0 = left ? i0 : j0;
#pragma unroll
    for (int u = 0; u < SQ; ++u) {
      const int e = tid + 256 * u;
      vS[u] = load4(Sb, r0 + e / 16, c0 + 4 * (e % 16), d);
    }
#pragma unroll
    for (int u = 0; u < AQ; ++u) {
      const int e = tid + 256 * u;
      vA[u] = load4(Pb, e / 16, j0 + 4 * (e % 16), r_a);
    }
  };
  load(0);
  for (int J = 0; J < nch; ++J) {
    __syncthreads();  // the previous chunk is no longer read
    const bool left = J < I;
#pragma unroll
    for (int u = 0; u < SQ; ++u) {
      const int e = tid + 256 * u, rr = e / 16, cc = 4 * (e % 16);
      const float v[4] = {vS[u].x, vS[u].y, vS[u].z, vS[u].w};
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        if (left) sS[(cc + q) * kPSL + rr] = v[q];
        else sS[rr * kPSL + cc + q] = v[q];
      }
    }
#pragma unroll
    for (int u = 0; u < AQ; ++u) {
      const int e = tid + 256 * u, a = e / 16, cc = 4 * (e % 16);
      sA[a * kPSL + cc] = vA[u].x;
      sA[a * kPSL + cc + 1] = vA[u].y;
      sA[a * kPSL + cc + 2] = vA[u].z;
      sA[a * kPSL + cc + 3] = vA[u].w;
    }
    if (J + 1 < nch) load(J + 1);  // in flight during this chunk's products
    __syncthreads();
    if (J == I) {  // diagonal chunk: only its upper triangle is stored; mirror it
#pragma unroll
      for (int u = 0; u < kPS * kPS / 256; ++u) {
        const int e = tid + 256 * u, rr = e / kPS, cc = e % kPS;
        if (cc < rr) sS[rr * kPSL + cc] = sS[cc * kPSL + rr];
      }
      __syncthreads();
    }
#pragma unroll
    for (int ks = 16 * w; ks < 16 * w + 16; ks += 2) {
      const int kk = ks + (lane >> 5);
      float fa[2], fb[NCB];
#pragma unroll
      for (int rb = 0; rb < 2; ++rb) fa[rb] = sS[(32 * rb + (lane & 31)) * kPSL + kk];
#pragma unroll
      for (int cb = 0; cb < NCB; ++cb) fb[cb] = sA[(32 * cb + (lane & 31)) * kPSL + kk];
#pragma unroll
      for (int rb = 0; rb < 2; ++rb)
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) acc[rb][cb] = mfma_f32x2(fa[rb], fb[cb], acc[rb][cb]);
    }
  }
#pragma unroll
  for (int rb = 0; rb < 2; ++rb)
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        sRed[w][32 * rb + mfma32_row(lane, r)][32 * cb + mfma32_col(lane)] = acc[rb][cb][r];
  __syncthreads();
  for (int e = tid; e < kPS * RA; e += 256) {
    const int rr = e / RA, a = e % RA;
    const int64_t i = i0 + rr;
    if (i < d && a < r_a)
      T1[(b * d + i) * r_a + a] =
          ((double)sRed[0][rr][a] + (double)sRed[1][rr][a]) + ((double)sRed[2][rr][a] + (double)sRed[3][rr][a]);
  }
}

// G[b] = PA T1 (r_a x r_a) and AK[b] = PA K (r_a x k), fp64, in two passes: partial sums
// over kProjSplit ranges of the rows (grid.z), then a fixed-order sum.  In the first, thread
// c of a workgroup takes column c of [T1 | K] and forms its entries for all RA rows of PA
// (RA sums in registers, rows a >= r_a zero); the rows of PA come 64 entries at a time
// through LDS, read four at a time by every thread alike (broadcast).
constexpr int kProjSplit = 64;
constexpr int kProjT = 192;  // threads: columns of [T1 | K] (r_a + k <= 64 + 128 by the API limits)
constexpr int kProjI = 64;   // rows of PA per LDS stage
template <typename ST, int RA>
__global__ __launch_bounds__(kProjT) void k_proj_small_part(int64_t d, int64_t k, int64_t r_a,
                                                            const float* __restrict__ PA, int64_t pa_bstride,
                                                            const double* __restrict__ T1, const ST* __restrict__ K,
                                                            int64_t k_bstride, double* __restrict__ part) {
  __shared__ __attribute__((aligned(16))) float sP[RA][kProjI];
  const int64_t b = blockIdx.y, z = blockIdx.z;
  const int64_t nout = r_a * r_a + r_a * k;
  const int c = (int)threadIdx.x;  // column of [T1 | K]
  const bool on = c < r_a + k;
  const int64_t chunk = (d + kProjSplit - 1) / kProjSplit;
  const int64_t i0 = z * chunk, i1 = i0 + chunk < d ? i0 + chunk : d;
  const float* P = PA + b * pa_bstride;
  const bool t1 = c < r_a;
  const double* T = T1 + b * d * r_a + (t1 ? c : 0);
  const ST* Kc = K + b * k_bstride + (t1 ? 0 : c - r_a);
  double s[RA];
#pragma unroll
  for (int a = 0; a < RA; ++a) s[a] = 0.0;
  for (int64_t is = i0; is < i1; is += kProjI) {
    const int ni = (int)(i1 - is < kProjI ? i1 - is : kProjI);
    __syncthreads();  // the previous stage is no longer read
    for (int e = c; e < RA * kProjI; e += kProjT) {
      const int a = e / kProjI, ii = e % kProjI;
      sP[a][ii] = (a < r_a && ii < ni) ? P[a * d + is + ii] : 0.f;
    }
    __syncthreads();
    if (on)
      for (int ii = 0; ii < ni; ii += 4) {
        double v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int64_t i = is + ii + u;
          v[u] = ii + u < ni ? (t1 ? T[i * r_a] : (double)Kc[i * k]) : 0.0;
        }
#pragma unroll
        for (int a = 0; a < RA; ++a) {
          const float4 p4 = *(const float4*)&sP[a][ii];
          s[a] += (double)p4.x * v[0];
          s[a] += (double)p4.y * v[1];
          s[a] += (double)p4.z * v[2];
          s[a] += (double)p4.w * v[3];
        }
      }
  }
  if (!on) return;
  double* out = part + (b * kProjSplit + z) * nout;
#pragma unroll
  for (int a = 0; a < RA; ++a) {
    if (a >= r_a) break;
    if (t1) out[a * r_a + c] = s[a];
    else out[r_a * r_a + a * k + (c - r_a)] = s[a];
  }
}
__global__ void k_proj_small_sum(int64_t k, int64_t r_a, const double* __restrict__ part, double* __restrict__ G,
                                 double* __restrict__ AK, float* __restrict__ g_out) {
  const int64_t b = blockIdx.y;
  const int64_t nout = r_a * r_a + r_a * k;
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= nout) return;
  double s = 0.0;
  for (int z = 0; z < kProjSplit; ++z) s += part[(b * kProjSplit + z) * nout + e];
  if (e < r_a * r_a) {
    G[b * r_a * r_a + e] = s;
    if (g_out) g_out[b * r_a * r_a + e] = (float)s;
  } else {
    AK[b * r_a * k + (e - r_a * r_a)] = s;
  }
}

// L = chol(G_b + lam_l I) once per (block, lambda), one wave (lower triangle, row-major
// r_a x r_a in Lw); a non-positive pivot goes to dev_info[mi] (1-based).
__global__ __launch_bounds__(64) void k_proj_chol(int64_t r_a, const double* __restrict__ G,
                                                  const double* __restrict__ lam, int nl, double* __restrict__ Lw,
                                                  int32_t* __restrict__ dev_info) {
  constexpr int LD = kMaxKp + 1;
  __shared__ double sL[kMaxKp * LD];
  const int64_t mi = blockIdx.x;
  const int64_t b = mi / nl;
  const int l = (int)(mi % nl);
  const int ra = (int)r_a, lane = threadIdx.x;
  for (int e = lane; e < ra * ra; e += 64) {
    const int i = e / ra, j = e % ra;
    sL[i * LD + j] = G[b * r_a * r_a + e] + (i == j ? lam[l] : 0.0);
  }
  __syncthreads();
  for (int j = 0; j < ra; ++j) {
    const double piv = sL[j * LD + j];
    if (lane == 0 && !(piv > 0.0)) atomicCAS(&dev_info[mi], 0, j + 1);
    const double ljj = sqrt(piv);
    __syncthreads();  // every lane has read the pivot
    if (lane == 0) sL[j * LD + j] = ljj;
    for (int i = j + 1 + lane; i < ra; i += 64) sL[i * LD + j] /= ljj;
    __syncthreads();
    for (int e = lane; e < (ra - j - 1) * (ra - j - 1); e += 64) {
      const int i = j + 1 + e / (ra - j - 1), c = j + 1 + e % (ra - j - 1);
      if (c <= i) sL[i * LD + c] -= sL[i * LD + j] * sL[c * LD + j];
    }
    __syncthreads();
  }
  for (int e = lane; e < ra * ra; e += 64) {
    const int i = e / ra, j = e % ra;
    Lw[mi * r_a * r_a + e] = j <= i ? sL[i * LD + j] : 0.0;
  }
}

// One thread per row i of B*: C[i] = B_cur[i] G + sum_c B~[c][i] AK[:, c], then the row
// solve x (L L^T) = C[i] (forward with L, backward with L^T), fp64, RA >= r_a registers.
// AK sits transposed in LDS ([c][a], zero for a >= r_a), read by every thread alike
// (broadcast); G and L are read at wave-uniform addresses.  The row of B* leaves in 16-byte
// stores when r_a % 4 == 0.
template <int RA>
__global__ __launch_bounds__(256) void k_proj_rows(int64_t d, int64_t k, int64_t r_a, const double* __restrict__ G,
                                                   const double* __restrict__ AK, const double* __restrict__ Lw,
                                                   const float* __restrict__ Bt, int64_t b_bstride,
                                                   const float* __restrict__ Bc, int64_t bc_bstride, int nl,
                                                   float* __restrict__ out, int64_t bo_bstride) {
  __shared__ __attribute__((aligned(16))) double sAK[128 * RA];  // [c][a], k <= 128
  const int64_t mi = blockIdx.y;
  const int64_t b = mi / nl;
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const bool ok = i < d;
  const int64_t ic = ok ? i : 0;
  const float* Btb = Bt + b * b_bstride;
  const double* AKb = AK + b * r_a * k;
  const double* L = Lw + mi * r_a * r_a;
  const int kk = (int)k;
  for (int e = threadIdx.x; e < kk * RA; e += 256) {
    const int c = e / RA, a = e % RA;
    sAK[e] = a < r_a ? AKb[a * k + c] : 0.0;
  }
  __syncthreads();
  double x[RA];
#pragma unroll
  for (int a = 0; a < RA; ++a) x[a] = 0.0;
  for (int c = 0; c < kk; ++c) {
    const double bt = (double)Btb[(int64_t)c * d + ic];
    const double* row = sAK + c * RA;
#pragma unroll
    for (int a = 0; a < RA; ++a) x[a] += bt * row[a];
  }
  if (Bc) {
    const float* Bci = Bc + b * bc_bstride + ic * r_a;
    const double* Gb = G + b * r_a * r_a;
    for (int64_t c = 0; c < r_a; ++c) {
      const double v = (double)Bci[c];
#pragma unroll
      for (int a = 0; a < RA; ++a)
        if (a < r_a) x[a] += v * Gb[c * r_a + a];
    }
  }
#pragma unroll
  for (int a = 0; a < RA; ++a) {  // forward: L y = c
    if (a < r_a) {
      double v = x[a];
#pragma unroll
      for (int c = 0; c < a; ++c) v -= L[a * r_a + c] * x[c];
      x[a] = v / L[a * r_a + a];
    }
  }
#pragma unroll
  for (int a = RA - 1; a >= 0; --a) {  // backward: L^T z = y
    if (a < r_a) {
      double v = x[a];
#pragma unroll
      for (int c = a + 1; c < RA; ++c)
        if (c < r_a) v -= L[c * r_a + a] * x[c];
      x[a] = v / L[a * r_a + a];
    }
  }
  if (ok) {
    float* o = out + mi * bo_bstride + i * r_a;
    if ((r_a & 3) == 0 && (bo_bstride & 3) == 0 && ((uintptr_t)out & 15) == 0) {
#pragma unroll
      for (int a = 0; a < RA; a += 4)
        if (a < r_a) *(float4*)(o + a) = make_float4((float)x[a], (float)x[a + 1], (float)x[a + 2], (float)x[a + 3]);
    } else {
#pragma unroll
      for (int a = 0; a < RA; ++a)
        if (a < r_a) o[a] = (float)x[a];
    }
  }
}

struct Lams8 {
  double v[8];
};
__global__ void k_set_lams8(Lams8 l, double* out, int cnt) {
  if ((int)threadIdx.x < cnt) out[threadIdx.x] = l.v[threadIdx.x];
}

}  // namespace

size_t projected_ws(int64_t nb, int64_t d, int64_t k, int64_t r_a, int64_t n_lambda) {
  size_t s = align256(sizeof(double) * nb * d * r_a);  // T1
  s += align256(sizeof(double) * nb * kProjSplit * (r_a * r_a + r_a * k));  // partials of G and AK
  s += align256(sizeof(double) * nb * r_a * r_a);      // G
  s += align256(sizeof(double) * nb * r_a * k);        // AK
  s += 256;                                            // lambdas
  s += align256(sizeof(double) * nb * (n_lambda > 0 ? n_lambda : 1) * r_a * r_a);  // Cholesky factors
  return s;
}

hipError_t launch_ridge_solve_projected(const ProjArgs& a) {
  char* p = a.ws;
  double* T1 = (double*)p; p += align256(sizeof(double) * a.nb * a.d * a.r_a);
  double* gpart = (double*)p; p += align256(sizeof(double) * a.nb * kProjSplit * (a.r_a * a.r_a + a.r_a * a.k));
  double* G = (double*)p; p += align256(sizeof(double) * a.nb * a.r_a * a.r_a);
  double* AK = (double*)p; p += align256(sizeof(double) * a.nb * a.r_a * a.k);
  double* dlam = (double*)p; p += 256;
  double* Lw = (double*)p;
  Lams8 l8;
  for (int i = 0; i < 8; ++i) l8.v[i] = (i < a.n_lambda) ? a.lambdas[i] : 0.0;
  k_set_lams8<<<1, 64, 0, a.stream>>>(l8, dlam, (int)a.n_lambda);
  const int64_t nm = a.nb * a.n_lambda;
  k_fill_zero<<<(unsigned)((nm + 255) / 256), 256, 0, a.stream>>>(a.dev_info, nm);
  dim3 g1((unsigned)((a.d * a.r_a + 255) / 256), (unsigned)a.nb);
  if (a.r_a + a.k > kProjT) return hipErrorInvalidValue;  // one thread per column of [T1 | K]
  dim3 g2(1u, (unsigned)a.nb, kProjSplit);
  if (a.acc == LOCA_F64) {
    k_proj_sa<double><<<g1, 256, 0, a.stream>>>(a.d, a.r_a, (const double*)a.S, a.s_bstride, a.proj_a, a.pa_bstride, T1);
    if (a.r_a <= 32)
      k_proj_small_part<double, 32><<<g2, kProjT, 0, a.stream>>>(a.d, a.k, a.r_a, a.proj_a, a.pa_bstride, T1,
                                                                  (const double*)a.K, a.k_bstride, gpart);
    else
      k_proj_small_part<double, 64><<<g2, kProjT, 0, a.stream>>>(a.d, a.k, a.r_a, a.proj_a, a.pa_bstride, T1,
                                                                  (const double*)a.K, a.k_bstride, gpart);
  } else {
    dim3 gp((unsigned)((a.d + kPS - 1) / kPS), (unsigned)a.nb);
    const float* Sf = (const float*)a.S;
    // 16-byte loads of S rows and PA rows need 16-byte aligned bases and strides
    const bool v4 = a.d % 4 == 0 && ((uintptr_t)Sf % 16) == 0 && ((uintptr_t)a.proj_a % 16) == 0 &&
                    a.s_bstride % 4 == 0 && a.pa_bstride % 4 == 0;
#define LOCA_PROJ_SA(RA, V)                                                                                   \
  k_proj_sa_mfma<RA, V><<<gp, 256, 0, a.stream>>>(a.d, a.r_a, Sf, a.s_bstride, a.proj_a, a.pa_bstride, T1)
    if (a.r_a <= 32) {
      if (v4) LOCA_PROJ_SA(32, true);
      else LOCA_PROJ_SA(32, false);
    } else {
      if (v4) LOCA_PROJ_SA(64, true);
      else LOCA_PROJ_SA(64, false);
    }
#undef LOCA_PROJ_SA
    if (a.r_a <= 32)
      k_proj_small_part<float, 32><<<g2, kProjT, 0, a.stream>>>(a.d, a.k, a.r_a, a.proj_a, a.pa_bstride, T1,
                                                                 (const float*)a.K, a.k_bstride, gpart);
    else
      k_proj_small_part<float, 64><<<g2, kProjT, 0, a.stream>>>(a.d, a.k, a.r_a, a.proj_a, a.pa_bstride, T1,
                                                                 (const float*)a.K, a.k_bstride, gpart);
  }
  dim3 g2s((unsigned)((a.r_a * a.r_a + a.r_a * a.k + 255) / 256), (unsigned)a.nb);
  k_proj_small_sum<<<g2s, 256, 0, a.stream>>>(a.k, a.r_a, gpart, G, AK, a.g_out);
  k_proj_chol<<<(unsigned)nm, 64, 0, a.stream>>>(a.r_a, G, dlam, (int)a.n_lambda, Lw, a.dev_info);
  dim3 g3((unsigned)((a.d + 255) / 256), (unsigned)nm);
#define LOCA_PROJ_ROWS(RA)                                                                                           \
  k_proj_rows<RA><<<g3, 256, 0, a.stream>>>(a.d, a.k, a.r_a, G, AK, Lw, a.credit_b, a.b_bstride, a.b_cur, a.bc_bstride, \
                                            (int)a.n_lambda, a.b_out, a.bo_bstride)
  if (a.r_a <= 16) LOCA_PROJ_ROWS(16);
  else if (a.r_a <= 32) LOCA_PROJ_ROWS(32);
  else LOCA_PROJ_ROWS(64);
#undef LOCA_PROJ_ROWS
  return hipGetLastError();
}

}  // namespace loca
