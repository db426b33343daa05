/*
 * sanitize_driver.c -- TEST INFRASTRUCTURE: drives every routine of loca_oracle.c
 * on small ragged shapes so that a host build with AddressSanitizer and
 * UndefinedBehaviorSanitizer (tests/test_oracle_sanitized.py) sees each of them
 * read and write its whole arrays.  Arrays are allocated at their exact sizes, so
 * any access past an end is reported.  Each check is a property the oracle's
 * pins also establish (row sums of the error, the normal-equation residual, the
 * reconstruction of a factorisation); the process exits non-zero on a failure.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

int loca_oracle_head_error(int64_t n, int64_t C, const double* z, const int32_t* y, const double* w, double* E);
void loca_oracle_credit(int64_t n, int64_t C, int64_t k, int64_t d, const double* E, const double* A,
                        const double* B, double* Y, double* Q);
void loca_oracle_scaled_target(int64_t n, int64_t d, const double* X, const double* Q, const double* a,
                               double eta, double* T, double* info);
void loca_oracle_gram_acc(int64_t n, int64_t d, const double* X, const double* a, double* S);
void loca_oracle_cross_acc(int64_t n, int64_t d, int64_t m, const double* X, const double* a, const double* T,
                           double* Z);
void loca_oracle_gram_entries(int64_t n, int64_t d, const double* X, int64_t npairs, const int64_t* ij,
                              double* out);
int loca_oracle_cholesky(int64_t d, double* A);
void loca_oracle_cholesky_solve(int64_t d, int64_t m, const double* L, double* B);
int loca_oracle_ridge_solve(int64_t d, int64_t m, const double* S, const double* RHS, double lam, double* W,
                            double* resid);
int loca_oracle_svd(int64_t rows, int64_t cols, const double* A, double* U, double* s, double* V);
int loca_oracle_truncate_dense(int64_t d, const double* W, int64_t r, double* W_r, double* sigma);
void loca_oracle_qr(int64_t rows, int64_t cols, const double* A, double* Q, double* R);
int loca_oracle_truncate_factored(int64_t d, int64_t kp, const double* M, const double* Rf, int64_t r,
                                  double* W_r, double* sigma, double* a_out, double* b_out);
void loca_oracle_projected_acc(int64_t n, int64_t d, int64_t r, const double* X, const double* T,
                               const double* Aproj, const double* Bcur, const double* a_w, double* G, double* Cst);
int loca_oracle_projected_solve(int64_t d, int64_t r, const double* G, const double* Cst, double lam,
                                double* Bstar, double* resid);

static uint64_t rng_state = 0x9E3779B97F4A7C15ull;
static double urand(void) { /* xorshift64*, uniform on (-1, 1) */
  rng_state ^= rng_state >> 12;
  rng_state ^= rng_state << 25;
  rng_state ^= rng_state >> 27;
  return (double)((rng_state * 2685821657736338717ull) >> 11) / 4503599627370496.0 - 1.0;
}
static double* vec(int64_t cnt) {
  double* p = (double*)malloc(sizeof(double) * (size_t)(cnt > 0 ? cnt : 1));
  for (int64_t i = 0; i < cnt; ++i) p[i] = urand();
  return p;
}
static int failures = 0;
static void check(int ok, const char* what) {
  if (!ok) {
    fprintf(stderr, "FAILED: %s\n", what);
    ++failures;
  }
}

int main(void) {
  const int64_t n = 37, C = 5, k = 3, d = 11, r = 4;
  double* z = vec(n * C);
  int32_t* y = (int32_t*)malloc(sizeof(int32_t) * n);
  for (int64_t t = 0; t < n; ++t) y[t] = (int32_t)(t % C);
  double* w = vec(n);
  double* E = vec(n * C);
  check(loca_oracle_head_error(n, C, z, y, w, E) == 0, "head_error status");
  for (int64_t t = 0; t < n; ++t) {
    double s = 0.0;
    for (int64_t c = 0; c < C; ++c) s += E[t * C + c];
    check(fabs(s) < 1e-12, "error rows sum to zero");
  }
  y[7] = (int32_t)C;
  check(loca_oracle_head_error(n, C, z, y, NULL, E) == -8, "bad label reported");
  y[7] = 2;

  double *A = vec(C * k), *B = vec(k * d), *Y = vec(n * k), *Q = vec(n * d), *X = vec(n * d), *T = vec(n * d);
  double* aw = vec(n);
  for (int64_t t = 0; t < n; ++t) aw[t] = fabs(aw[t]);
  loca_oracle_credit(n, C, k, d, E, A, B, Y, Q);
  double info[3];
  loca_oracle_scaled_target(n, d, X, Q, aw, 0.01, T, info);
  check(info[0] > 0.0 && info[1] > 0.0 && info[2] > 0.0, "scaled target");

  double *S = (double*)calloc((size_t)(d * d), sizeof(double)), *Z = (double*)calloc((size_t)(d * k), sizeof(double));
  loca_oracle_gram_acc(n, d, X, aw, S);
  loca_oracle_cross_acc(n, d, k, X, aw, Y, Z);
  int64_t ij[6] = {0, 0, 3, 10, 10, 4};
  double ent[3];
  loca_oracle_gram_entries(n, d, X, 3, ij, ent);
  check(isfinite(ent[0] + ent[1] + ent[2]), "gram entries");

  double* W = vec(d * k);
  double resid = 1.0;
  check(loca_oracle_ridge_solve(d, k, S, Z, 0.1, W, &resid) == 0 && resid < 1e-10, "ridge solve residual");
  double* L = vec(d * d);
  for (int64_t i = 0; i < d * d; ++i) L[i] = S[i] + (i % (d + 1) == 0 ? 0.1 : 0.0);
  check(loca_oracle_cholesky(d, L) == 0, "cholesky");
  double* Bs = vec(d * 2);
  loca_oracle_cholesky_solve(d, 2, L, Bs);

  const int64_t rows = 9, cols = 6;
  double *M = vec(rows * cols), *U = vec(rows * cols), *sv = vec(cols), *V = vec(cols * cols);
  check(loca_oracle_svd(rows, cols, M, U, sv, V) > 0, "svd sweeps");
  for (int64_t j = 1; j < cols; ++j) check(sv[j - 1] >= sv[j], "singular values decrease");
  double *Qm = vec(rows * cols), *Rm = vec(cols * cols);
  loca_oracle_qr(rows, cols, M, Qm, Rm);
  for (int64_t i = 0; i < rows; ++i)
    for (int64_t j = 0; j < cols; ++j) {
      double v = 0.0;
      for (int64_t p = 0; p < cols; ++p) v += Qm[i * cols + p] * Rm[p * cols + j];
      check(fabs(v - M[i * cols + j]) < 1e-12, "QR reconstructs");
    }

  double *Wd = vec(d * d), *Wr = vec(d * d), *sg = vec(d);
  check(loca_oracle_truncate_dense(d, Wd, 3, Wr, sg) > 0, "dense truncation");
  double *Mf = vec(d * k), *Rf = vec(k * d), *Wr2 = vec(d * d), *sg2 = vec(k), *ao = vec(r * d), *bo = vec(d * r);
  check(loca_oracle_truncate_factored(d, k, Mf, Rf, r, Wr2, sg2, ao, bo) > 0, "factored truncation (r > kp)");

  double *Ap = vec(r * d), *Bc = vec(d * r), *G = (double*)calloc((size_t)(r * r), sizeof(double));
  double* Cst = (double*)calloc((size_t)(d * r), sizeof(double));
  loca_oracle_projected_acc(n, d, r, X, T, Ap, Bc, aw, G, Cst);
  double* Bstar = vec(d * r);
  check(loca_oracle_projected_solve(d, r, G, Cst, 0.5, Bstar, &resid) == 0 && resid < 1e-10, "projected solve");

  free(z); free(y); free(w); free(E); free(A); free(B); free(Y); free(Q); free(X); free(T); free(aw);
  free(S); free(Z); free(W); free(L); free(Bs); free(M); free(U); free(sv); free(V); free(Qm); free(Rm);
  free(Wd); free(Wr); free(sg); free(Mf); free(Rf); free(Wr2); free(sg2); free(ao); free(bo);
  free(Ap); free(Bc); free(G); free(Cst); free(Bstar);
  if (failures) return 1;
  printf("sanitized oracle driver: ok\n");
  return 0;
}
