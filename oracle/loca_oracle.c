/*
 * loca_oracle.c -- plain float64 reference for the LoCA per-block adaptation
 * step.  TEST INFRASTRUCTURE ONLY: it is built and called by the test suite,
 * by the package's smoke check and by the benchmark's CPU-baseline leg, never
 * by the HIP path, and it shares no code with it.
 *
 * Every routine is the textbook definition written out with plain loops in
 * float64, row-major arrays, no blocking and no algebraic shortcuts: the
 * hidden-state target T and the cross statistic Z = X^T T are materialised
 * densely, the ridge system is solved by an unblocked Cholesky, and the
 * truncation uses an explicit one-sided Jacobi SVD.  OpenMP only splits
 * independent output rows between threads; each output element is summed in
 * the same order whatever the thread count.
 *
 * Notation (paper): X (N x d) holds the block inputs h_{l-1} at the selected
 * positions, one token per row; E (N x C) the head error rows; A~ (C x k) and
 * B~ (k x d) the low-rank credit factors with the head folded into A~, so that
 * the tokenwise feedback F_l e_t of Section S3 is the row Y_t B~ with Y = E A~.
 *
 * Pins: every function here is checked by the CPU tests against closed forms,
 * invariants, brute force or an independent library routine (numpy's SVD and
 * least squares); no function is "parity unpinned".
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define IDX(i, j, ld) ((size_t)(i) * (size_t)(ld) + (size_t)(j))

/* ------------------------------------------------------------------------
 * Lemma S3.1 (top-layer error) and the error in Eq. (4): the derivative of the
 * weighted cross-entropy at position t with respect to the logits is
 * w_t (softmax(z_t) - onehot(y_t)).  The frozen head W_u^T that maps it to the
 * hidden width is folded into the credit factor A~.  A zero weight gives a
 * zero row.  Softmax is evaluated with the row maximum subtracted.
 * Returns 0, or -(t+1) for the first row whose label is outside [0, C).
 * ------------------------------------------------------------------------ */
int loca_oracle_head_error(int64_t n, int64_t C, const double* z, const int32_t* y,
                           const double* w, double* E) {
  for (int64_t t = 0; t < n; ++t)
    if (y[t] < 0 || y[t] >= C) return (int)-(t + 1);
#pragma omp parallel for schedule(static)
  for (int64_t t = 0; t < n; ++t) {
    const double* zt = z + IDX(t, 0, C);
    double m = zt[0];
    for (int64_t c = 1; c < C; ++c)
      if (zt[c] > m) m = zt[c];
    double s = 0.0;
    for (int64_t c = 0; c < C; ++c) s += exp(zt[c] - m);
    const double wt = w ? w[t] : 1.0;
    for (int64_t c = 0; c < C; ++c) {
      double p = exp(zt[c] - m) / s;
      E[IDX(t, c, C)] = wt * (p - (c == y[t] ? 1.0 : 0.0));
    }
  }
  return 0;
}

/* ------------------------------------------------------------------------
 * Tokenwise feedback Q_l = F_l E (Section S3), applied through the rank-k
 * factors in the order of the cost model of Section S11, F_l e =
 * U_k (Sigma_k (V_k^T e)).  In row form: Y = E A~ (N x k), Q = Y B~ (N x d).
 * ------------------------------------------------------------------------ */
void loca_oracle_credit(int64_t n, int64_t C, int64_t k, int64_t d, const double* E,
                        const double* A, const double* B, double* Y, double* Q) {
#pragma omp parallel for schedule(static)
  for (int64_t t = 0; t < n; ++t)
    for (int64_t j = 0; j < k; ++j) {
      double s = 0.0;
      for (int64_t c = 0; c < C; ++c) s += E[IDX(t, c, C)] * A[IDX(c, j, k)];
      Y[IDX(t, j, k)] = s;
    }
  if (!Q) return;
#pragma omp parallel for schedule(static)
  for (int64_t t = 0; t < n; ++t)
    for (int64_t i = 0; i < d; ++i) {
      double s = 0.0;
      for (int64_t j = 0; j < k; ++j) s += Y[IDX(t, j, k)] * B[IDX(j, i, d)];
      Q[IDX(t, i, d)] = s;
    }
}

/* ------------------------------------------------------------------------
 * Scale-normalised target of one mini-batch (Eq. 10; Section S8):
 *   RMS(M) = ||M||_F / sqrt(#entries),
 *   eta_bar = eta * RMS(X) / RMS(Q)  if Q != 0, and 0 if Q = 0,
 *   D^tar  = -eta_bar Q            (the displacement; row t is T_t).
 * X and Q have the same shape (n x d).  With position weights a (n entries,
 * NULL = all ones; the weighted statistics of Section S7) every mean square is
 * taken under the same weights, RMS_a(M)^2 = sum_t a_t ||M_t||^2 / (d sum_t a_t),
 * so a position of weight 0 has no influence.
 * info = {sum_t a_t ||X_t||^2, sum_t a_t ||Q_t||^2, eta_bar}.
 * ------------------------------------------------------------------------ */
void loca_oracle_scaled_target(int64_t n, int64_t d, const double* X, const double* Q,
                               const double* a, double eta, double* T, double* info) {
  double sx = 0.0, sq = 0.0, wsum = 0.0;
  for (int64_t t = 0; t < n; ++t) {
    const double at = a ? a[t] : 1.0;
    double xt = 0.0, qt = 0.0;
    for (int64_t i = 0; i < d; ++i) {
      xt += X[IDX(t, i, d)] * X[IDX(t, i, d)];
      qt += Q[IDX(t, i, d)] * Q[IDX(t, i, d)];
    }
    sx += at * xt;
    sq += at * qt;
    wsum += at;
  }
  const double cnt = wsum * (double)d;
  double eta_bar = 0.0;
  if (sq > 0.0) eta_bar = eta * (sqrt(sx / cnt) / sqrt(sq / cnt));
  if (T)
    for (int64_t t = 0; t < n; ++t)
      for (int64_t i = 0; i < d; ++i) T[IDX(t, i, d)] = -eta_bar * Q[IDX(t, i, d)];
  info[0] = sx;
  info[1] = sq;
  info[2] = eta_bar;
}

/* ------------------------------------------------------------------------
 * Streaming sufficient statistics (Eq. 9; Section S7), additive over
 * mini-batches.  With the identity projection the features are the block
 * inputs themselves, so, with explicit nonnegative position weights a_t
 * (NULL = all ones),
 *   S += sum_t a_t x_t x_t^T          (d x d, full square),
 *   Z += sum_t a_t x_t T_t^T          (d x m) for a target block T (n x m).
 * ------------------------------------------------------------------------ */
void loca_oracle_gram_acc(int64_t n, int64_t d, const double* X, const double* a, double* S) {
#pragma omp parallel for schedule(dynamic, 4)
  for (int64_t i = 0; i < d; ++i)
    for (int64_t j = 0; j < d; ++j) {
      double s = 0.0;
      for (int64_t t = 0; t < n; ++t) s += (a ? a[t] : 1.0) * X[IDX(t, i, d)] * X[IDX(t, j, d)];
      S[IDX(i, j, d)] += s;
    }
}

void loca_oracle_cross_acc(int64_t n, int64_t d, int64_t m, const double* X, const double* a,
                           const double* T, double* Z) {
#pragma omp parallel for schedule(dynamic, 4)
  for (int64_t i = 0; i < d; ++i)
    for (int64_t j = 0; j < m; ++j) {
      double s = 0.0;
      for (int64_t t = 0; t < n; ++t) s += (a ? a[t] : 1.0) * X[IDX(t, i, d)] * T[IDX(t, j, m)];
      Z[IDX(i, j, m)] += s;
    }
}

/* Entries S[i][j] = sum_t X[t][i] X[t][j] for a list of (i, j) pairs. */
void loca_oracle_gram_entries(int64_t n, int64_t d, const double* X, int64_t npairs,
                              const int64_t* ij, double* out) {
  for (int64_t p = 0; p < npairs; ++p) {
    const int64_t i = ij[2 * p], j = ij[2 * p + 1];
    double s = 0.0;
    for (int64_t t = 0; t < n; ++t) s += X[IDX(t, i, d)] * X[IDX(t, j, d)];
    out[p] = s;
  }
}

/* ------------------------------------------------------------------------
 * Cholesky factorisation A = L L^T of a symmetric positive-definite matrix
 * (textbook column-by-column Cholesky-Crout).  In place: on return the lower
 * triangle of A holds L and the strict upper triangle is zeroed.  Returns 0,
 * or the 1-based index of the first pivot that is not positive.
 * ------------------------------------------------------------------------ */
int loca_oracle_cholesky(int64_t d, double* A) {
  for (int64_t j = 0; j < d; ++j) {
    double s = A[IDX(j, j, d)];
    for (int64_t p = 0; p < j; ++p) s -= A[IDX(j, p, d)] * A[IDX(j, p, d)];
    if (!(s > 0.0)) return (int)(j + 1);
    const double ljj = sqrt(s);
    A[IDX(j, j, d)] = ljj;
#pragma omp parallel for schedule(static)
    for (int64_t i = j + 1; i < d; ++i) {
      double v = A[IDX(i, j, d)];
      for (int64_t p = 0; p < j; ++p) v -= A[IDX(i, p, d)] * A[IDX(j, p, d)];
      A[IDX(i, j, d)] = v / ljj;
    }
  }
  for (int64_t i = 0; i < d; ++i)
    for (int64_t j = i + 1; j < d; ++j) A[IDX(i, j, d)] = 0.0;
  return 0;
}

/* Solve L L^T X = B for m right-hand sides (B is d x m, overwritten by X).  The
 * right-hand sides are independent: OpenMP gives whole columns to threads. */
void loca_oracle_cholesky_solve(int64_t d, int64_t m, const double* L, double* B) {
#pragma omp parallel for schedule(static)
  for (int64_t c = 0; c < m; ++c) {
    for (int64_t i = 0; i < d; ++i) { /* forward: L y = b */
      double v = B[IDX(i, c, m)];
      for (int64_t p = 0; p < i; ++p) v -= L[IDX(i, p, d)] * B[IDX(p, c, m)];
      B[IDX(i, c, m)] = v / L[IDX(i, i, d)];
    }
    for (int64_t i = d - 1; i >= 0; --i) { /* backward: L^T x = y */
      double v = B[IDX(i, c, m)];
      for (int64_t p = i + 1; p < d; ++p) v -= L[IDX(p, i, d)] * B[IDX(p, c, m)];
      B[IDX(i, c, m)] = v / L[IDX(i, i, d)];
    }
  }
}

/* ------------------------------------------------------------------------
 * Ridge solve of Theorem S6.1 in the linear-system form of Section S7:
 *   (S + lam I) W = RHS     (S: d x d symmetric, full square; RHS: d x m),
 * by Cholesky, followed by one step of iterative refinement.  resid (may be
 * NULL) receives ||(S + lam I) W - RHS||_F / ||RHS||_F.  Returns 0 or the
 * failing pivot of the factorisation.
 * ------------------------------------------------------------------------ */
int loca_oracle_ridge_solve(int64_t d, int64_t m, const double* S, const double* RHS, double lam,
                            double* W, double* resid) {
  double* L = (double*)malloc(sizeof(double) * (size_t)d * (size_t)d);
  double* R = (double*)malloc(sizeof(double) * (size_t)d * (size_t)m);
  if (!L || !R) { free(L); free(R); return -1; }
  for (int64_t i = 0; i < d; ++i)
    for (int64_t j = 0; j < d; ++j) L[IDX(i, j, d)] = S[IDX(i, j, d)] + (i == j ? lam : 0.0);
  int info = loca_oracle_cholesky(d, L);
  if (info) { free(L); free(R); return info; }
  memcpy(W, RHS, sizeof(double) * (size_t)d * (size_t)m);
  loca_oracle_cholesky_solve(d, m, L, W);
  /* refinement: R = RHS - (S + lam I) W ; W += solve(R) */
  for (int pass = 0; pass < 2; ++pass) {
    double num = 0.0, den = 0.0;
#pragma omp parallel for schedule(static) reduction(+ : num, den)
    for (int64_t i = 0; i < d; ++i)
      for (int64_t c = 0; c < m; ++c) {
        double v = RHS[IDX(i, c, m)];
        for (int64_t j = 0; j < d; ++j) v -= S[IDX(i, j, d)] * W[IDX(j, c, m)];
        v -= lam * W[IDX(i, c, m)];
        R[IDX(i, c, m)] = v;
        num += v * v;
        den += RHS[IDX(i, c, m)] * RHS[IDX(i, c, m)];
      }
    if (pass == 1) {
      if (resid) *resid = den > 0.0 ? sqrt(num / den) : sqrt(num);
      break;
    }
    loca_oracle_cholesky_solve(d, m, L, R);
    for (size_t e = 0; e < (size_t)d * (size_t)m; ++e) W[e] += R[e];
  }
  free(L);
  free(R);
  return 0;
}

/* ------------------------------------------------------------------------
 * Singular value decomposition A = U diag(s) V^T of a rows x cols matrix with
 * rows >= cols by one-sided Jacobi (Hestenes): plane rotations orthogonalise
 * pairs of columns until every pair is orthogonal to working precision.
 * U is rows x cols, V is cols x cols, s has cols entries sorted in decreasing
 * order.  Columns with zero singular value get a zero U column.
 * Returns the number of sweeps used (or -1 on allocation failure).
 * ------------------------------------------------------------------------ */
int loca_oracle_svd(int64_t rows, int64_t cols, const double* A, double* U, double* s, double* V) {
  /* column-major working copies: a[j*rows + i] = A[i][j] */
  double* a = (double*)malloc(sizeof(double) * (size_t)rows * (size_t)cols);
  double* v = (double*)malloc(sizeof(double) * (size_t)cols * (size_t)cols);
  double* nrm = (double*)malloc(sizeof(double) * (size_t)cols);
  int64_t* ord = (int64_t*)malloc(sizeof(int64_t) * (size_t)cols);
  if (!a || !v || !nrm || !ord) { free(a); free(v); free(nrm); free(ord); return -1; }
  for (int64_t i = 0; i < rows; ++i)
    for (int64_t j = 0; j < cols; ++j) a[(size_t)j * rows + i] = A[IDX(i, j, cols)];
  for (int64_t i = 0; i < cols; ++i)
    for (int64_t j = 0; j < cols; ++j) v[(size_t)j * cols + i] = (i == j) ? 1.0 : 0.0;
  const double eps = 1e-15;
  int sweep;
  for (sweep = 1; sweep <= 60; ++sweep) {
    int64_t rotated = 0;
    for (int64_t p = 0; p < cols - 1; ++p)
      for (int64_t q = p + 1; q < cols; ++q) {
        double* ap = a + (size_t)p * rows;
        double* aq = a + (size_t)q * rows;
        double alpha = 0.0, beta = 0.0, gamma = 0.0;
        for (int64_t i = 0; i < rows; ++i) {
          alpha += ap[i] * ap[i];
          beta += aq[i] * aq[i];
          gamma += ap[i] * aq[i];
        }
        if (gamma == 0.0 || fabs(gamma) <= eps * sqrt(alpha * beta)) continue;
        ++rotated;
        const double zeta = (beta - alpha) / (2.0 * gamma);
        const double tt = (zeta >= 0.0 ? 1.0 : -1.0) / (fabs(zeta) + sqrt(1.0 + zeta * zeta));
        const double c = 1.0 / sqrt(1.0 + tt * tt), sn = c * tt;
        for (int64_t i = 0; i < rows; ++i) {
          const double x = ap[i], y = aq[i];
          ap[i] = c * x - sn * y;
          aq[i] = sn * x + c * y;
        }
        double* vp = v + (size_t)p * cols;
        double* vq = v + (size_t)q * cols;
        for (int64_t i = 0; i < cols; ++i) {
          const double x = vp[i], y = vq[i];
          vp[i] = c * x - sn * y;
          vq[i] = sn * x + c * y;
        }
      }
    if (!rotated) break;
  }
  for (int64_t j = 0; j < cols; ++j) {
    double t = 0.0;
    for (int64_t i = 0; i < rows; ++i) t += a[(size_t)j * rows + i] * a[(size_t)j * rows + i];
    nrm[j] = sqrt(t);
    ord[j] = j;
  }
  /* sort by decreasing singular value (insertion sort, stable) */
  for (int64_t i = 1; i < cols; ++i) {
    int64_t key = ord[i], j = i - 1;
    while (j >= 0 && nrm[ord[j]] < nrm[key]) { ord[j + 1] = ord[j]; --j; }
    ord[j + 1] = key;
  }
  for (int64_t jj = 0; jj < cols; ++jj) {
    const int64_t j = ord[jj];
    s[jj] = nrm[j];
    for (int64_t i = 0; i < rows; ++i)
      U[IDX(i, jj, cols)] = nrm[j] > 0.0 ? a[(size_t)j * rows + i] / nrm[j] : 0.0;
    for (int64_t i = 0; i < cols; ++i) V[IDX(i, jj, cols)] = v[(size_t)j * cols + i];
  }
  free(a); free(v); free(nrm); free(ord);
  return sweep;
}

/* ------------------------------------------------------------------------
 * Best rank-r approximation (Lemma S5.2, Eckart-Young), applied to the dense
 * ridge solution W (d x d): W_r = sum_{j<r} s_j u_j v_j^T.  sigma receives all d
 * singular values.  Explicit SVD of the dense matrix.
 * ------------------------------------------------------------------------ */
int loca_oracle_truncate_dense(int64_t d, const double* W, int64_t r, double* W_r, double* sigma) {
  double* U = (double*)malloc(sizeof(double) * (size_t)d * (size_t)d);
  double* V = (double*)malloc(sizeof(double) * (size_t)d * (size_t)d);
  if (!U || !V) { free(U); free(V); return -1; }
  int sw = loca_oracle_svd(d, d, W, U, sigma, V);
  for (int64_t i = 0; i < d; ++i)
    for (int64_t j = 0; j < d; ++j) {
      double t = 0.0;
      for (int64_t p = 0; p < r && p < d; ++p) t += U[IDX(i, p, d)] * sigma[p] * V[IDX(j, p, d)];
      W_r[IDX(i, j, d)] = t;
    }
  free(U); free(V);
  return sw;
}

/* ------------------------------------------------------------------------
 * Householder QR of a rows x cols matrix (rows >= cols): A = Q R with Q
 * (rows x cols) having orthonormal columns and R (cols x cols) upper
 * triangular.  Rank-deficient inputs are fine (R gets zero diagonal entries).
 * ------------------------------------------------------------------------ */
void loca_oracle_qr(int64_t rows, int64_t cols, const double* A, double* Q, double* R) {
  double* a = (double*)malloc(sizeof(double) * (size_t)rows * (size_t)cols);
  double* vs = (double*)malloc(sizeof(double) * (size_t)rows * (size_t)cols);
  double* beta = (double*)malloc(sizeof(double) * (size_t)cols);
  memcpy(a, A, sizeof(double) * (size_t)rows * (size_t)cols);
  for (int64_t j = 0; j < cols; ++j) {
    double* v = vs + (size_t)j * rows;
    double nx = 0.0;
    for (int64_t i = j; i < rows; ++i) nx += a[IDX(i, j, cols)] * a[IDX(i, j, cols)];
    nx = sqrt(nx);
    for (int64_t i = 0; i < rows; ++i) v[i] = (i >= j) ? a[IDX(i, j, cols)] : 0.0;
    if (nx == 0.0) { beta[j] = 0.0; continue; }
    const double alpha = (a[IDX(j, j, cols)] >= 0.0) ? -nx : nx;
    v[j] -= alpha;
    double vv = 0.0;
    for (int64_t i = j; i < rows; ++i) vv += v[i] * v[i];
    beta[j] = (vv > 0.0) ? 2.0 / vv : 0.0;
    for (int64_t c = j; c < cols; ++c) { /* a <- (I - beta v v^T) a */
      double t = 0.0;
      for (int64_t i = j; i < rows; ++i) t += v[i] * a[IDX(i, c, cols)];
      t *= beta[j];
      for (int64_t i = j; i < rows; ++i) a[IDX(i, c, cols)] -= t * v[i];
    }
  }
  for (int64_t i = 0; i < cols; ++i)
    for (int64_t j = 0; j < cols; ++j) R[IDX(i, j, cols)] = (j >= i) ? a[IDX(i, j, cols)] : 0.0;
  /* Q = H_0 H_1 ... H_{cols-1} [I; 0] */
  for (int64_t i = 0; i < rows; ++i)
    for (int64_t j = 0; j < cols; ++j) Q[IDX(i, j, cols)] = (i == j) ? 1.0 : 0.0;
  for (int64_t j = cols - 1; j >= 0; --j) {
    const double* v = vs + (size_t)j * rows;
    if (beta[j] == 0.0) continue;
    for (int64_t c = 0; c < cols; ++c) {
      double t = 0.0;
      for (int64_t i = j; i < rows; ++i) t += v[i] * Q[IDX(i, c, cols)];
      t *= beta[j];
      for (int64_t i = j; i < rows; ++i) Q[IDX(i, c, cols)] -= t * v[i];
    }
  }
  free(a); free(vs); free(beta);
}

/* ------------------------------------------------------------------------
 * Eckart-Young truncation (Lemma S5.2) of a ridge solution known in factored
 * form W = M R (M: d x kp, R: kp x d), for widths where a dense d x d SVD is
 * too slow.  Thin QR M = Q_m R_m, then the SVD of the small factor
 * C^T = (R_m R)^T = U_c diag(s) V_c^T gives W = (Q_m V_c) diag(s) U_c^T exactly.
 * Outputs: W_r (d x d, may be NULL), sigma (kp values), the adapter factors
 * a_out = (Q_m V_c)[:, :r]^T (r x d) and b_out = U_c[:, :r] diag(s_r) (d x r),
 * so that W_r = a_out^T b_out^T (either may be NULL).  Requires kp <= d.
 * ------------------------------------------------------------------------ */
int loca_oracle_truncate_factored(int64_t d, int64_t kp, const double* M, const double* Rf,
                                  int64_t r, double* W_r, double* sigma, double* a_out,
                                  double* b_out) {
  double* Q = (double*)malloc(sizeof(double) * (size_t)d * (size_t)kp);
  double* Rm = (double*)malloc(sizeof(double) * (size_t)kp * (size_t)kp);
  double* Ct = (double*)malloc(sizeof(double) * (size_t)d * (size_t)kp);
  double* Uc = (double*)malloc(sizeof(double) * (size_t)d * (size_t)kp);
  double* Vc = (double*)malloc(sizeof(double) * (size_t)kp * (size_t)kp);
  double* L = (double*)malloc(sizeof(double) * (size_t)d * (size_t)kp);
  loca_oracle_qr(d, kp, M, Q, Rm);
  for (int64_t i = 0; i < d; ++i) /* Ct[i][a] = sum_b Rm[a][b] Rf[b][i] */
    for (int64_t a = 0; a < kp; ++a) {
      double t = 0.0;
      for (int64_t b = 0; b < kp; ++b) t += Rm[IDX(a, b, kp)] * Rf[IDX(b, i, d)];
      Ct[IDX(i, a, kp)] = t;
    }
  int sw = loca_oracle_svd(d, kp, Ct, Uc, sigma, Vc);
  for (int64_t i = 0; i < d; ++i) /* left singular vectors L = Q Vc */
    for (int64_t a = 0; a < kp; ++a) {
      double t = 0.0;
      for (int64_t b = 0; b < kp; ++b) t += Q[IDX(i, b, kp)] * Vc[IDX(b, a, kp)];
      L[IDX(i, a, kp)] = t;
    }
  const int64_t rr = r < kp ? r : kp;
  if (W_r)
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < d; ++i)
      for (int64_t j = 0; j < d; ++j) {
        double t = 0.0;
        for (int64_t p = 0; p < rr; ++p) t += L[IDX(i, p, kp)] * sigma[p] * Uc[IDX(j, p, kp)];
        W_r[IDX(i, j, d)] = t;
      }
  if (a_out)
    for (int64_t p = 0; p < r; ++p)
      for (int64_t i = 0; i < d; ++i) a_out[IDX(p, i, d)] = (p < rr) ? L[IDX(i, p, kp)] : 0.0;
  if (b_out)
    for (int64_t i = 0; i < d; ++i)
      for (int64_t p = 0; p < r; ++p) b_out[IDX(i, p, r)] = (p < rr) ? Uc[IDX(i, p, kp)] * sigma[p] : 0.0;
  free(Q); free(Rm); free(Ct); free(Uc); free(Vc); free(L);
  return sw;
}

/* ------------------------------------------------------------------------
 * Paper-literal projected statistics (Eqs. 6 and 9; Section S6), streamed over
 * a mini-batch: with p_t = A_l x_t (A_l: r x d fixed random projection) and
 * residual target rho_t = B_cur p_t + T_t (B_cur: d x r current adapter, may be
 * NULL for the frozen model) and nonnegative position weights a_t (NULL = 1;
 * the weighted form of Section S7),
 *   G += sum_t a_t p_t p_t^T   (r x r),     Cst += sum_t a_t rho_t p_t^T   (d x r).
 * ------------------------------------------------------------------------ */
void loca_oracle_projected_acc(int64_t n, int64_t d, int64_t r, const double* X, const double* T,
                               const double* Aproj, const double* Bcur, const double* a_w, double* G,
                               double* Cst) {
  double* P = (double*)malloc(sizeof(double) * (size_t)n * (size_t)r);
  double* Rho = (double*)malloc(sizeof(double) * (size_t)n * (size_t)d);
#pragma omp parallel for schedule(static)
  for (int64_t t = 0; t < n; ++t)
    for (int64_t a = 0; a < r; ++a) {
      double s = 0.0;
      for (int64_t i = 0; i < d; ++i) s += Aproj[IDX(a, i, d)] * X[IDX(t, i, d)];
      P[IDX(t, a, r)] = s;
    }
#pragma omp parallel for schedule(static)
  for (int64_t t = 0; t < n; ++t)
    for (int64_t i = 0; i < d; ++i) {
      double s = T[IDX(t, i, d)];
      if (Bcur)
        for (int64_t a = 0; a < r; ++a) s += Bcur[IDX(i, a, r)] * P[IDX(t, a, r)];
      Rho[IDX(t, i, d)] = s;
    }
  for (int64_t a = 0; a < r; ++a)
    for (int64_t b = 0; b < r; ++b) {
      double s = 0.0;
      for (int64_t t = 0; t < n; ++t) s += (a_w ? a_w[t] : 1.0) * P[IDX(t, a, r)] * P[IDX(t, b, r)];
      G[IDX(a, b, r)] += s;
    }
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < d; ++i)
    for (int64_t a = 0; a < r; ++a) {
      double s = 0.0;
      for (int64_t t = 0; t < n; ++t) s += (a_w ? a_w[t] : 1.0) * Rho[IDX(t, i, d)] * P[IDX(t, a, r)];
      Cst[IDX(i, a, r)] += s;
    }
  free(P);
  free(Rho);
}

/* Closed-form block minimiser (Eq. 7; Theorem S6.1): B* = Cst (G + lam I)^{-1},
 * solved as (G + lam I) B*^T = Cst^T (Section S7).  B* is d x r. */
int loca_oracle_projected_solve(int64_t d, int64_t r, const double* G, const double* Cst, double lam,
                                double* Bstar, double* resid) {
  double* Ct = (double*)calloc((size_t)r * (size_t)d, sizeof(double));
  double* Xs = (double*)calloc((size_t)r * (size_t)d, sizeof(double));
  if (!Ct || !Xs) { free(Ct); free(Xs); return -1; }
  for (int64_t i = 0; i < d; ++i)
    for (int64_t a = 0; a < r; ++a) Ct[IDX(a, i, d)] = Cst[IDX(i, a, r)];
  int info = loca_oracle_ridge_solve(r, d, G, Ct, lam, Xs, resid);
  if (!info)
    for (int64_t i = 0; i < d; ++i)
      for (int64_t a = 0; a < r; ++a) Bstar[IDX(i, a, r)] = Xs[IDX(a, i, d)];
  free(Ct);
  free(Xs);
  return info;
}
