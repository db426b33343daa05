"""Pins of the float64 oracle against what the paper and the mathematics fix.

None of these re-types the oracle's own formula: each checks a closed form, an
invariant, a special case, brute force, or an independent library routine
(numpy/LAPACK), chosen so that a dropped term, a wrong sign or index or a
transposed operand in the oracle fails at least one of them.
"""
import json
import os

import numpy as np
import pytest

HERE = os.path.dirname(os.path.abspath(__file__))


def rel(a, b):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    den = np.linalg.norm(b)
    return np.linalg.norm(a - b) / (den if den > 0 else 1.0)


def ce_loss(z, y):
    m = z.max()
    return -z[y] + m + np.log(np.exp(z - m).sum())


# ------------------------------------------------------------------ head error (Lemma S3.1)


@pytest.mark.parametrize("C", [1, 2, 5, 37])
def test_head_error_is_gradient_of_ce(orc, C):
    """E_t = w_t dCE/dz_t: checked by central finite differences of the loss."""
    rng = np.random.default_rng(C)
    n = 7
    z = rng.normal(0, 2, (n, C))
    y = rng.integers(0, C, n)
    w = rng.uniform(0.2, 2.0, n)
    E = orc.head_error(z, y, w)
    h = 1e-6
    for t in range(n):
        for c in range(C):
            zp, zm = z[t].copy(), z[t].copy()
            zp[c] += h
            zm[c] -= h
            fd = w[t] * (ce_loss(zp, y[t]) - ce_loss(zm, y[t])) / (2 * h)
            assert abs(E[t, c] - fd) < 1e-7


def test_head_error_invariants(orc):
    rng = np.random.default_rng(1)
    z = rng.normal(0, 3, (50, 6))
    y = rng.integers(0, 6, 50)
    w = np.ones(50)
    w[::7] = 0.0
    E = orc.head_error(z, y, w)
    assert np.max(np.abs(E.sum(axis=1))) < 1e-14          # rows sum to zero
    assert np.all(E[::7] == 0.0)                            # zero-weight positions give e_t = 0
    # the label entry is the only negative one (p - 1 < 0), others are probabilities
    for t in range(50):
        if w[t] > 0:
            assert E[t, y[t]] < 0 and np.all(np.delete(E[t], y[t]) > 0)
    # C = 1: softmax is 1, so the error vanishes
    assert np.all(orc.head_error(rng.normal(size=(4, 1)), np.zeros(4, np.int32)) == 0.0)


def test_head_error_two_class_closed_form(orc):
    """C = 2: E_t1 = sigmoid(z1 - z0) - [y = 1] = -E_t0."""
    z = np.array([[0.0, np.log(3.0)], [1.5, -0.5], [-2.0, 2.0]])
    y = np.array([0, 1, 1], np.int32)
    E = orc.head_error(z, y)
    sig = 1.0 / (1.0 + np.exp(-(z[:, 1] - z[:, 0])))
    np.testing.assert_allclose(E[:, 1], sig - (y == 1), rtol=0, atol=1e-15)
    np.testing.assert_allclose(E[:, 0], -E[:, 1], rtol=0, atol=1e-15)
    # hand value: z = (0, ln 3), y = 0 -> p = (1/4, 3/4), E = (-3/4, 3/4)
    np.testing.assert_allclose(E[0], [-0.75, 0.75], atol=1e-15)


def test_head_error_rejects_bad_label(orc):
    with pytest.raises(ValueError):
        orc.head_error(np.zeros((3, 4)), np.array([0, 4, 1], np.int32))


# ------------------------------------------------------------------ credit map (Section S3, S11)


def test_credit_matches_paper_factorisation(orc):
    """q_t = F_l e_t with F_l = U_k S_k V_k^T and e_t = W_u^T E_t (Eq. 4, Sections S5, S11).

    The oracle takes the folded factors A~ = W_u V_k and B~ = S_k U_k^T; the
    test builds F_l and e_t from the paper's objects and compares.
    """
    rng = np.random.default_rng(2)
    n, C, d, k = 9, 11, 13, 4
    Wu = rng.normal(size=(C, d))                      # frozen head, V x d
    U, _ = np.linalg.qr(rng.normal(size=(d, k)))
    V, _ = np.linalg.qr(rng.normal(size=(d, k)))
    Sk = np.diag(np.sort(rng.uniform(0.5, 3.0, k))[::-1])
    F = U @ Sk @ V.T                                  # d x d, rank k
    z = rng.normal(size=(n, C))
    y = rng.integers(0, C, n)
    E = orc.head_error(z, y)
    A = Wu @ V                                        # C x k
    B = Sk @ U.T                                      # k x d
    Y, Q = orc.credit(E, A, B)
    for t in range(n):
        e_t = Wu.T @ E[t]                             # hidden-width top error
        np.testing.assert_allclose(Q[t], F @ e_t, rtol=0, atol=1e-12)
        np.testing.assert_allclose(Y[t], V.T @ e_t, rtol=0, atol=1e-12)


def test_credit_all_ones_column_is_zero(orc):
    rng = np.random.default_rng(3)
    E = orc.head_error(rng.normal(size=(20, 5)), rng.integers(0, 5, 20))
    A = rng.normal(size=(5, 3))
    A[:, 1] = 1.0
    Y, _ = orc.credit(E, A, rng.normal(size=(3, 8)))
    assert np.max(np.abs(Y[:, 1])) < 1e-15


# ------------------------------------------------------------------ scale-normalised target (Eq. 10, S8)


def test_target_rms_identity_and_scale_invariance(orc):
    rng = np.random.default_rng(4)
    X = rng.normal(size=(30, 17)) * 3
    Q = rng.normal(size=(30, 17))
    eta = 0.03
    T, info = orc.scaled_target(X, Q, eta)
    rms = lambda M: np.sqrt(np.mean(M ** 2))
    assert abs(rms(T) - eta * rms(X)) < 1e-14 * rms(X)          # Proposition S8.1
    T2, _ = orc.scaled_target(X, 7.5 * Q, eta)
    np.testing.assert_allclose(T2, T, rtol=1e-14, atol=1e-16)    # positive scale invariance
    # direction is -Q
    assert np.all(np.sign(T[Q != 0]) == -np.sign(Q[Q != 0]))
    assert abs(info["sum_x2"] - np.sum(X ** 2)) < 1e-10 * np.sum(X ** 2)


def test_target_zero_feedback(orc):
    X = np.ones((4, 3))
    T, info = orc.scaled_target(X, np.zeros((4, 3)), 0.01)
    assert info["eta_bar"] == 0.0 and np.all(T == 0.0)


# ------------------------------------------------------------------ statistics (Eq. 9, S7)


def test_gram_cross_against_library_and_invariants(orc):
    rng = np.random.default_rng(5)
    X = rng.normal(size=(40, 12))
    T = rng.normal(size=(40, 12))
    S = orc.gram_acc(X)
    Z = orc.cross_acc(X, T)
    np.testing.assert_allclose(S, X.T @ X, rtol=1e-13, atol=1e-12)   # BLAS as independent check
    np.testing.assert_allclose(Z, X.T @ T, rtol=1e-13, atol=1e-12)
    assert abs(np.trace(S) - np.sum(X ** 2)) < 1e-12 * np.sum(X ** 2)
    assert np.array_equal(S, S.T)
    assert np.min(np.linalg.eigvalsh(S)) > -1e-10
    # orientation: with one-hot rows, S counts and Z copies targets
    Xe = np.zeros((3, 4))
    Xe[0, 1] = Xe[1, 1] = Xe[2, 3] = 1.0
    Te = np.arange(12.0).reshape(3, 4)
    Se = orc.gram_acc(Xe)
    assert Se[1, 1] == 2 and Se[3, 3] == 1 and Se.sum() == 3
    Ze = orc.cross_acc(Xe, Te)
    np.testing.assert_array_equal(Ze[1], Te[0] + Te[1])
    np.testing.assert_array_equal(Ze[3], Te[2])


def test_matmul_statistics_equal_plain_loops(orc):
    """The library-product forms used at full workload width (gram_matmul, cross_matmul,
    credit_matmul) against the plain loops pinned above, with and without weights; and the
    one-hot orientation check on the product forms themselves."""
    rng = np.random.default_rng(55)
    X = rng.normal(size=(37, 11))
    T = rng.normal(size=(37, 5))
    a = rng.uniform(0.0, 2.0, 37)
    a[::4] = 0.0
    np.testing.assert_allclose(orc.gram_matmul(X), orc.gram_acc(X), rtol=1e-13, atol=1e-12)
    np.testing.assert_allclose(orc.gram_matmul(X, a), orc.gram_acc(X, a=a), rtol=1e-13, atol=1e-12)
    np.testing.assert_allclose(orc.cross_matmul(X, T), orc.cross_acc(X, T), rtol=1e-13, atol=1e-12)
    np.testing.assert_allclose(orc.cross_matmul(X, T, a), orc.cross_acc(X, T, a=a), rtol=1e-13, atol=1e-12)
    E = orc.head_error(rng.normal(0, 2, (37, 6)), rng.integers(0, 6, 37))
    A = rng.normal(size=(6, 4))
    B = rng.normal(size=(4, 11))
    Y, Q = orc.credit(E, A, B)
    Ym, Qm = orc.credit_matmul(E, A, B)
    np.testing.assert_allclose(Ym, Y, rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(Qm, Q, rtol=1e-13, atol=1e-13)
    Xe = np.zeros((3, 4))
    Xe[0, 1] = Xe[1, 1] = Xe[2, 3] = 1.0
    Se = orc.gram_matmul(Xe)
    assert Se[1, 1] == 2 and Se[3, 3] == 1 and Se.sum() == 3
    Te = np.arange(12.0).reshape(3, 4)
    np.testing.assert_array_equal(orc.cross_matmul(Xe, Te)[1], Te[0] + Te[1])


def test_streaming_additivity(orc):
    """Section S7: statistics over the concatenation equal the sum over mini-batches."""
    rng = np.random.default_rng(6)
    X1, X2 = rng.normal(size=(17, 9)), rng.normal(size=(23, 9))
    T1, T2 = rng.normal(size=(17, 9)), rng.normal(size=(23, 9))
    S = orc.gram_acc(X2, orc.gram_acc(X1))
    Z = orc.cross_acc(X2, T2, orc.cross_acc(X1, T1))
    np.testing.assert_allclose(S, orc.gram_acc(np.vstack([X1, X2])), rtol=1e-13)
    np.testing.assert_allclose(Z, orc.cross_acc(np.vstack([X1, X2]), np.vstack([T1, T2])), rtol=1e-13)


def test_gram_entries(orc):
    rng = np.random.default_rng(7)
    X = rng.normal(size=(33, 10))
    pairs = np.array([[0, 0], [3, 7], [9, 2], [5, 5]])
    v = orc.gram_entries(X, pairs)
    for p, (i, j) in enumerate(pairs):
        assert abs(v[p] - np.dot(X[:, i], X[:, j])) < 1e-12


# ------------------------------------------------------------------ Cholesky and ridge solve (Thm S6.1, S7)


def test_cholesky_against_lapack(orc):
    rng = np.random.default_rng(8)
    M = rng.normal(size=(25, 25))
    A = M @ M.T + 0.5 * np.eye(25)
    L = orc.cholesky(A)
    np.testing.assert_allclose(L, np.linalg.cholesky(A), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(L @ L.T, A, rtol=1e-13, atol=1e-12)
    bad = A.copy()
    bad[4, 4] = -1.0
    with pytest.raises(np.linalg.LinAlgError):
        orc.cholesky(bad)


def _ridge_problem(rng, n, d, m):
    X = rng.normal(size=(n, d)) * rng.uniform(0.3, 5, d)
    T = rng.normal(size=(n, m))
    return X, T, X.T @ X, X.T @ T


@pytest.mark.parametrize("n,d", [(1, 4), (3, 8), (17, 8), (64, 33), (8, 33)])
def test_ridge_brute_force_augmented_lstsq(orc, n, d):
    """W = argmin ||X W - T||^2 + lam ||W||^2 equals least squares on [X; sqrt(lam) I]."""
    rng = np.random.default_rng(n * 100 + d)
    lam = 0.37
    X, T, S, Z = _ridge_problem(rng, n, d, d)
    W, resid = orc.ridge_solve(S, Z, lam)
    Xa = np.vstack([X, np.sqrt(lam) * np.eye(d)])
    Ta = np.vstack([T, np.zeros((d, d))])
    Wls = np.linalg.lstsq(Xa, Ta, rcond=None)[0]
    assert rel(W, Wls) < 1e-10
    assert resid <= 1e-10


def test_ridge_dual_form_when_n_below_d(orc):
    """Push-through identity (Section S5 uses it for the feedback fit): for N < d,
    (X^T X + lam I_d)^{-1} X^T T = X^T (X X^T + lam I_N)^{-1} T."""
    rng = np.random.default_rng(9)
    X, T, S, Z = _ridge_problem(rng, 12, 40, 40)
    lam = 1e-2
    W, _ = orc.ridge_solve(S, Z, lam)
    Wd = X.T @ np.linalg.solve(X @ X.T + lam * np.eye(12), T)
    assert rel(W, Wd) < 1e-9


def test_ridge_gap_identity(orc):
    """Theorem S6.1: Phi(B) - Phi(B*) = tr((B - B*)(G + lam I)(B - B*)^T) for any B."""
    rng = np.random.default_rng(10)
    X, T, S, Z = _ridge_problem(rng, 30, 10, 6)
    lam = 0.8
    W, _ = orc.ridge_solve(S, Z, lam)
    phi = lambda Wm: np.sum((X @ Wm - T) ** 2) + lam * np.sum(Wm ** 2)
    for _ in range(3):
        Wb = W + rng.normal(size=W.shape)
        D = Wb - W
        gap = np.trace(D.T @ (S + lam * np.eye(10)) @ D)
        assert abs((phi(Wb) - phi(W)) - gap) < 1e-9 * max(1.0, gap)
        assert phi(Wb) > phi(W)


def test_realization_error_pins(orc):
    """Section S6's realisation error E_fit = X (W - W_prev) - T, pinned by consequences of
    Theorem S6.1 rather than by its own formula:
      * first-order condition at the ridge solution: X^T E_fit = -lam W;
      * the ridge objective fit2 + lam w2 is the residual of the augmented least-squares
        problem [X; sqrt(lam) I] W = [X W_prev + T; 0] solved by LAPACK;
      * no change (W = W_prev) realises nothing: fit2 = tar2;
      * a target inside the feature span (T = X V) is realised exactly as lam -> 0;
      * position weights scale each row's contribution."""
    rng = np.random.default_rng(31)
    n, d, m = 40, 9, 9
    X = rng.normal(size=(n, d)) * rng.uniform(0.5, 3, d)
    T = rng.normal(size=(n, m))
    Wp = 0.3 * rng.normal(size=(d, m))
    lam = 0.7
    S = X.T @ X
    W, _ = orc.ridge_solve(S, S @ Wp + X.T @ T, lam)
    r = orc.realization_error(X, T, W, Wp, want_e=True)
    np.testing.assert_allclose(X.T @ r["E"], -lam * W, atol=1e-10 * np.abs(W).max() * lam)
    aug_X = np.vstack([X, np.sqrt(lam) * np.eye(d)])
    aug_T = np.vstack([X @ Wp + T, np.zeros((d, m))])
    Wl, res, _, _ = np.linalg.lstsq(aug_X, aug_T, rcond=None)
    np.testing.assert_allclose(W, Wl, rtol=1e-9, atol=1e-12)
    assert abs((r["fit2"] + lam * r["w2"]) - res.sum()) < 1e-9 * res.sum()
    assert abs(r["tar2"] - np.sum(T * T)) < 1e-12 * r["tar2"]
    r0 = orc.realization_error(X, T, Wp, Wp)
    assert abs(r0["fit2"] - r0["tar2"]) < 1e-12 * r0["tar2"]
    V = rng.normal(size=(d, m))
    Ts = X @ V
    Ws, _ = orc.ridge_solve(S, X.T @ Ts, 1e-10)
    assert orc.realization_error(X, Ts, Ws)["fit2"] < 1e-12 * np.sum(Ts * Ts)
    a = rng.uniform(0, 2, n)
    a[3] = 0.0
    ra = orc.realization_error(X, T, W, Wp, a=a, want_e=True)
    assert abs(ra["fit2"] - np.sum(a * np.sum(ra["E"] ** 2, axis=1))) < 1e-12 * ra["fit2"]
    Xd = X.copy()
    Xd[3] *= 100.0  # a zero-weight row has no influence
    Td = T.copy()
    Td[3] += 5.0
    assert abs(orc.realization_error(Xd, Td, W, Wp, a=a)["fit2"] - ra["fit2"]) < 1e-12 * ra["fit2"]


def test_ridge_limits(orc):
    rng = np.random.default_rng(11)
    X, T, S, Z = _ridge_problem(rng, 50, 7, 3)
    W_big, _ = orc.ridge_solve(S, Z, 1e12)
    assert np.linalg.norm(W_big) < 1e-8 * np.linalg.norm(Z)           # W -> 0
    assert rel(1e12 * W_big, Z) < 1e-6                                  # lam W -> Z
    W_small, _ = orc.ridge_solve(S, Z, 1e-12)
    W_ols = np.linalg.lstsq(X, T, rcond=None)[0]                        # full column rank, N >= d
    assert rel(W_small, W_ols) < 1e-8


def test_ridge_nonpd_reports(orc):
    with pytest.raises(np.linalg.LinAlgError):
        orc.ridge_solve(-np.eye(3), np.ones((3, 1)), 0.5)


# ------------------------------------------------------------------ SVD and truncation (Lemma S5.2)


@pytest.mark.parametrize("rows,cols", [(6, 6), (20, 7), (33, 33)])
def test_svd_against_lapack(orc, rows, cols):
    rng = np.random.default_rng(rows + cols)
    A = rng.normal(size=(rows, cols))
    U, s, V = orc.svd(A)
    np.testing.assert_allclose(s, np.linalg.svd(A, compute_uv=False), rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(U * s @ V.T, A, atol=1e-12)
    np.testing.assert_allclose(U.T @ U, np.eye(cols), atol=1e-12)
    np.testing.assert_allclose(V.T @ V, np.eye(cols), atol=1e-12)


def test_qr(orc):
    rng = np.random.default_rng(12)
    A = rng.normal(size=(15, 6))
    A[:, 4] = A[:, 1] * 2.0                      # rank-deficient column
    Q, R = orc.qr(A)
    np.testing.assert_allclose(Q @ R, A, atol=1e-12)
    np.testing.assert_allclose(Q.T @ Q, np.eye(6), atol=1e-12)
    assert np.allclose(np.tril(R, -1), 0.0)


def test_truncation_eckart_young(orc):
    rng = np.random.default_rng(13)
    d, r = 24, 5
    W = rng.normal(size=(d, d))
    Wr, s = orc.truncate_dense(W, r)
    s_np = np.linalg.svd(W, compute_uv=False)
    np.testing.assert_allclose(s, s_np, rtol=1e-12)
    assert abs(np.linalg.norm(W - Wr) ** 2 - np.sum(s_np[r:] ** 2)) < 1e-10 * np.sum(s_np ** 2)
    assert abs(np.linalg.norm(W - Wr, 2) - s_np[r]) < 1e-10 * s_np[0]
    U, sv, Vt = np.linalg.svd(W)
    np.testing.assert_allclose(Wr, (U[:, :r] * sv[:r]) @ Vt[:r], atol=1e-11)
    assert np.linalg.matrix_rank(Wr, tol=1e-9) == r


def test_truncation_factored_equals_dense(orc):
    rng = np.random.default_rng(14)
    d, kp, r = 40, 9, 4
    M = rng.normal(size=(d, kp))
    R = rng.normal(size=(kp, d))
    W = M @ R
    Wr_d, s_d = orc.truncate_dense(W, r)
    Wr_f, s_f, a, b = orc.truncate_factored(M, R, r)
    np.testing.assert_allclose(s_f, s_d[:kp], rtol=1e-11, atol=1e-12 * s_d[0])
    assert np.all(s_d[kp:] < 1e-10 * s_d[0])
    assert rel(Wr_f, Wr_d) < 1e-11
    np.testing.assert_allclose(a.T @ b.T, Wr_f, atol=1e-11)             # adapter factors reproduce W_r
    np.testing.assert_allclose(a @ a.T, np.eye(r), atol=1e-12)           # A = U_r^T has orthonormal rows
    # rank-deficient M (rank 2 < kp): truncation to r >= rank returns W exactly
    M2 = rng.normal(size=(d, 2)) @ rng.normal(size=(2, kp))
    Wr2, s2, _, _ = orc.truncate_factored(M2, R, r)
    assert rel(Wr2, M2 @ R) < 1e-11 and np.all(s2[2:] < 1e-10 * s2[0])


# ------------------------------------------------------------------ projected form (Eqs. 6-9)


def test_projected_statistics_identities(orc):
    """G_l = A_l S A_l^T and C_l = B_cur G_l + Z^T A_l^T with p = A_l x (derived from Eq. 9)."""
    rng = np.random.default_rng(15)
    n, d, r = 40, 12, 3
    X, T = rng.normal(size=(n, d)), rng.normal(size=(n, d))
    Ap = rng.normal(size=(r, d)) / np.sqrt(d)
    Bc = rng.normal(size=(d, r))
    G, Cst = orc.projected_acc(X, T, Ap, Bc)
    S, Z = orc.gram_acc(X), orc.cross_acc(X, T)
    np.testing.assert_allclose(G, Ap @ S @ Ap.T, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(Cst, Bc @ G + Z.T @ Ap.T, rtol=1e-12, atol=1e-11)
    # closed form B* = C (G + lam I)^{-1}: first-order condition B* (G + lam I) = C
    Bs, resid = orc.projected_solve(G, Cst, 0.3)
    np.testing.assert_allclose(Bs @ (G + 0.3 * np.eye(r)), Cst, atol=1e-10)
    assert resid < 1e-12


def test_projected_identity_projection_is_dense_solve(orc):
    """A_l = I_d turns the paper's block fit into the full-width one: B* = W^T."""
    rng = np.random.default_rng(16)
    n, d = 25, 8
    X, T = rng.normal(size=(n, d)), rng.normal(size=(n, d))
    G, Cst = orc.projected_acc(X, T, np.eye(d))
    Bs, _ = orc.projected_solve(G, Cst, 0.05)
    W, _ = orc.ridge_solve(orc.gram_acc(X), orc.cross_acc(X, T), 0.05)
    assert rel(Bs, W.T) < 1e-11


# ------------------------------------------------------------------ one block, end to end


def _tiny_block(rng, n_mb=3, rows=(11, 20, 7), d=10, C=4, k=3):
    xs = [rng.normal(size=(r, d)) for r in rows[:n_mb]]
    zs = [rng.normal(0, 2, (r, C)) for r in rows[:n_mb]]
    ys = [rng.integers(0, C, r) for r in rows[:n_mb]]
    A = rng.normal(size=(C, k)) / np.sqrt(k)
    B = rng.normal(size=(k, d)) / np.sqrt(k)
    return xs, zs, ys, A, B


def test_block_step_consistency(orc):
    rng = np.random.default_rng(17)
    xs, zs, ys, A, B = _tiny_block(rng)
    out = orc.block_step(xs, zs, ys, A, B, 0.01, [1e-2, 1.0], r_a=2, Aproj=np.eye(10))
    # Z = K B~ (the cross statistic factors through the rank-k credit coordinates)
    assert rel(out["Z"], out["K"] @ B) < 1e-12
    for sol in out["solves"]:
        assert sol["resid"] <= 1e-10
        assert rel(sol["W"], sol["M"] @ B) < 1e-10
        assert rel(sol["B_proj"], sol["W"].T) < 1e-10
        # rank W <= min(k, C - 1): here C - 1 = 3 = k, r_a = 2 truncates
        s = sol["sigma"]
        assert np.all(s[3:] < 1e-9 * s[0])
    # each mini-batch's displacement has RMS eta * RMS(X_m)
    for X, T in zip(xs, out["T"]):
        assert abs(np.sqrt(np.mean(T ** 2)) - 0.01 * np.sqrt(np.mean(X ** 2))) < 1e-14


def test_block_step_rank_bound_two_classes(orc):
    """C = 2 makes every error row a multiple of (-1, 1): rank W <= 1 (frozen start)."""
    rng = np.random.default_rng(18)
    xs, zs, ys, A, B = _tiny_block(rng, C=2, k=5)
    out = orc.block_step(xs, zs, ys, A, B, 0.01, [1e-2], r_a=3)
    s = out["solves"][0]["sigma"]
    assert s[0] > 0 and np.all(s[1:] < 1e-10 * s[0])
    assert rel(out["solves"][0]["W_r"], out["solves"][0]["W"]) < 1e-10


def test_block_step_zero_eta_is_frozen_model(orc):
    """eta = 0 gives a zero target and a zero adapter: B = 0 recovers the frozen model."""
    rng = np.random.default_rng(19)
    xs, zs, ys, A, B = _tiny_block(rng)
    out = orc.block_step(xs, zs, ys, A, B, 0.0, [1e-2], r_a=2)
    assert np.all(out["solves"][0]["W"] == 0.0)


def test_block_step_current_adapter(orc):
    """Residual target rho = B_cur p - eta_bar q (Eq. 6): with zero target the solve
    shrinks the current adapter, W = (S + lam I)^{-1} S W_prev."""
    rng = np.random.default_rng(20)
    xs, zs, ys, A, B = _tiny_block(rng)
    Wp = rng.normal(size=(10, 10))
    out = orc.block_step(xs, zs, ys, A, B, 0.0, [0.5], r_a=2, W_prev=Wp)
    X = np.vstack(xs)
    W_ls = np.linalg.lstsq(np.vstack([X, np.sqrt(0.5) * np.eye(10)]),
                           np.vstack([X @ Wp, np.zeros((10, 10))]), rcond=None)[0]
    assert rel(out["solves"][0]["W"], W_ls) < 1e-10


# ------------------------------------------------------------------ golden fixture (hand-derived)


def test_golden_hand_example(orc):
    with open(os.path.join(HERE, "golden", "hand_example.json")) as f:
        g = json.load(f)
    X = np.array(g["X"], float)
    z = np.array(g["logits"], float)
    y = np.array(g["labels"], np.int32)
    A = np.array(g["A"], float)
    B = np.array(g["B"], float)
    out = orc.block_step([X], [z], [y], A, B, g["eta"], [g["lam"]], r_a=1)
    np.testing.assert_allclose(out["E"][0], np.array(g["E"]), atol=1e-15)
    np.testing.assert_allclose(out["mb"][0]["eta_bar"], g["eta_bar"], rtol=1e-14)
    np.testing.assert_allclose(out["T"][0], np.array(g["T"]), rtol=1e-13, atol=1e-16)
    np.testing.assert_allclose(out["S"], np.array(g["S"]), atol=1e-15)
    np.testing.assert_allclose(out["solves"][0]["W"], np.array(g["W"]), rtol=1e-13, atol=1e-16)
