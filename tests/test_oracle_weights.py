"""Pins of the oracle's weighted statistics (Section S7: explicit nonnegative
position weights a_n in G, C and the ridge objective) and of the weighted
scale normalisation (Eq. 10 under the same weights).  Each check compares with
an unweighted computation on a transformed data set, or with a brute-force
least-squares solve of the weighted objective, never with the weighted formula
retyped."""
from __future__ import annotations

import numpy as np


def _data(rng, n, d, m):
    X = rng.standard_normal((n, d))
    T = rng.standard_normal((n, m))
    return X, T


def test_integer_weights_repeat_rows(orc):
    # a_t in {0, 1, 2, 3}: the weighted statistics are those of X with row t repeated a_t times
    rng = np.random.default_rng(11)
    n, d, m = 23, 9, 4
    X, T = _data(rng, n, d, m)
    Q = rng.standard_normal((n, d))
    a = rng.integers(0, 4, n).astype(np.float64)
    a[3] = 0.0
    rep = np.repeat(np.arange(n), a.astype(int))
    np.testing.assert_allclose(orc.gram_acc(X, a=a), orc.gram_acc(X[rep]), rtol=1e-13, atol=1e-12)
    np.testing.assert_allclose(orc.cross_acc(X, T, a=a), orc.cross_acc(X[rep], T[rep]), rtol=1e-13, atol=1e-12)
    _, iw = orc.scaled_target(X, Q, 0.01, a)
    _, ir = orc.scaled_target(X[rep], Q[rep], 0.01)
    for key in ("sum_x2", "sum_q2", "eta_bar"):
        assert abs(iw[key] - ir[key]) <= 1e-13 * abs(ir[key]), key
    # the paper-literal projected statistics under the same weights
    r = 3
    Ap = rng.standard_normal((r, d)) / np.sqrt(d)
    Bc = rng.standard_normal((d, r))
    Tq = rng.standard_normal((n, d))
    Gw, Cw = orc.projected_acc(X, Tq, Ap, Bc, a=a)
    Gr, Cr = orc.projected_acc(X[rep], Tq[rep], Ap, Bc)
    np.testing.assert_allclose(Gw, Gr, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(Cw, Cr, rtol=1e-12, atol=1e-12)


def test_zero_weight_drops_the_position(orc):
    # a_t = 0 removes position t from S, Z and both mean squares (its values are irrelevant)
    rng = np.random.default_rng(12)
    n, d = 17, 6
    X, T = _data(rng, n, d, 3)
    Q = rng.standard_normal((n, d))
    a = np.ones(n)
    a[[0, 5, 16]] = 0.0
    keep = a > 0
    X2, Q2 = X.copy(), Q.copy()
    X2[~keep] *= 1e3     # the dropped rows may hold anything
    Q2[~keep] = 0.0
    np.testing.assert_allclose(orc.gram_acc(X2, a=a), orc.gram_acc(X[keep]), rtol=1e-13, atol=1e-12)
    np.testing.assert_allclose(orc.cross_acc(X2, T, a=a), orc.cross_acc(X[keep], T[keep]), rtol=1e-13, atol=1e-12)
    _, iw = orc.scaled_target(X2, Q2, 0.02, a)
    _, ir = orc.scaled_target(X[keep], Q[keep], 0.02)
    assert abs(iw["eta_bar"] - ir["eta_bar"]) <= 1e-13 * ir["eta_bar"]


def test_weighted_ridge_objective_brute_force(orc):
    # (S_a + lam I)^{-1} Z_a minimises sum_t a_t ||W^T x_t - T_t||^2 + lam ||W||_F^2:
    # least squares on the stacked system [sqrt(a) X; sqrt(lam) I] W = [sqrt(a) T; 0]
    rng = np.random.default_rng(13)
    n, d, m, lam = 40, 8, 5, 0.3
    X, T = _data(rng, n, d, m)
    a = rng.uniform(0.0, 2.0, n)
    W, _ = orc.ridge_solve(orc.gram_acc(X, a=a), orc.cross_acc(X, T, a=a), lam)
    sa = np.sqrt(a)[:, None]
    Aug = np.vstack([sa * X, np.sqrt(lam) * np.eye(d)])
    Rhs = np.vstack([sa * T, np.zeros((d, m))])
    W_ls = np.linalg.lstsq(Aug, Rhs, rcond=None)[0]
    np.testing.assert_allclose(W, W_ls, rtol=1e-10, atol=1e-12)


def test_constant_weight_rescales_lambda(orc):
    # a_t = c for all t: S and Z scale by c, eta_bar is unchanged, and the solve at
    # lam equals the unweighted solve at lam / c
    rng = np.random.default_rng(14)
    n, d, m, c, lam = 30, 7, 3, 2.5, 0.4
    X, T = _data(rng, n, d, m)
    Q = rng.standard_normal((n, d))
    a = np.full(n, c)
    _, iw = orc.scaled_target(X, Q, 0.01, a)
    _, iu = orc.scaled_target(X, Q, 0.01)
    assert abs(iw["eta_bar"] - iu["eta_bar"]) <= 1e-14 * iu["eta_bar"]
    Ww, _ = orc.ridge_solve(orc.gram_acc(X, a=a), orc.cross_acc(X, T, a=a), lam)
    Wu, _ = orc.ridge_solve(orc.gram_acc(X), orc.cross_acc(X, T), lam / c)
    np.testing.assert_allclose(Ww, Wu, rtol=1e-11, atol=1e-13)


def test_block_step_with_integer_weights_is_repetition(orc):
    # the whole block step with integer statistic weights equals the unweighted step on
    # the repeated rows (every micro-batch; factored and dense truncation alike)
    rng = np.random.default_rng(15)
    d, C, k, r_a = 12, 4, 3, 2
    A = rng.standard_normal((C, k)) / np.sqrt(k)
    B = rng.standard_normal((k, d)) / np.sqrt(k)
    xs, zs, ys, aws = [], [], [], []
    for n in (20, 13):
        xs.append(rng.standard_normal((n, d)))
        zs.append(rng.standard_normal((n, C)) * 2)
        ys.append(rng.integers(0, C, n))
        aws.append(rng.integers(0, 3, n).astype(np.float64))
    reps = [np.repeat(np.arange(len(a)), a.astype(int)) for a in aws]
    out_w = orc.block_step(xs, zs, ys, A, B, 0.01, [0.05], r_a, a_ws=aws)
    out_r = orc.block_step([x[r] for x, r in zip(xs, reps)], [z[r] for z, r in zip(zs, reps)],
                           [y[r] for y, r in zip(ys, reps)], A, B, 0.01, [0.05], r_a)
    for key in ("S", "Z", "K"):
        np.testing.assert_allclose(out_w[key], out_r[key], rtol=1e-12, atol=1e-12)
    for mw, mr in zip(out_w["mb"], out_r["mb"]):
        assert abs(mw["eta_bar"] - mr["eta_bar"]) <= 1e-13 * mr["eta_bar"]
    sw, sr = out_w["solves"][0], out_r["solves"][0]
    np.testing.assert_allclose(sw["M"], sr["M"], rtol=1e-10, atol=1e-13)
    np.testing.assert_allclose(sw["W_r"], sr["W_r"], rtol=1e-9, atol=1e-13)
