"""Pins of the oracle's Stage I calibration (Section S5): the feedback ridge fit, its
rank-k truncation, the credit factors and the alignment diagnostic, each checked
against a fact of the mathematics rather than against the oracle's own formula."""
from __future__ import annotations

import numpy as np
import pytest


def _pairs(rng, d, n_p, noise=0.0, rank=None):
    E = rng.standard_normal((d, n_p))
    F0 = rng.standard_normal((d, d)) / np.sqrt(d)
    if rank is not None:
        F0 = rng.standard_normal((d, rank)) @ rng.standard_normal((rank, d)) / d
    G = F0 @ E + noise * rng.standard_normal((d, n_p))
    return E, G, F0


def _objective(F, E, G, beta):
    return float(np.sum((F @ E - G) ** 2) + beta * np.sum(F ** 2))


@pytest.mark.parametrize("d,n_p", [(30, 12), (12, 30), (24, 24)])
def test_primal_and_dual_agree(orc, d, n_p):
    # push-through identity: E^T (E E^T + b I_d)^{-1} = (E^T E + b I_Np)^{-1} E^T
    rng = np.random.default_rng(1)
    E, G, _ = _pairs(rng, d, n_p, noise=0.1)
    Fd = orc.feedback_fit(E, G, 0.05, "dual")
    Fp = orc.feedback_fit(E, G, 0.05, "primal")
    np.testing.assert_allclose(Fd, Fp, rtol=1e-10, atol=1e-12)


def test_first_order_condition_and_optimality(orc):
    rng = np.random.default_rng(2)
    d, n_p, beta = 20, 35, 0.3
    E, G, _ = _pairs(rng, d, n_p, noise=0.5)
    F = orc.feedback_fit(E, G, beta)
    # gradient of the objective vanishes: (F E - G) E^T + beta F = 0
    grad = (F @ E - G) @ E.T + beta * F
    assert np.abs(grad).max() < 1e-10 * max(1.0, np.abs(G @ E.T).max())
    # strictly convex: every perturbation raises the objective by ||D E||^2 + beta ||D||^2
    f0 = _objective(F, E, G, beta)
    for _ in range(5):
        D = 1e-3 * rng.standard_normal(F.shape)
        gain = _objective(F + D, E, G, beta) - f0
        expect = np.sum((D @ E) ** 2) + beta * np.sum(D ** 2)
        assert gain > 0 and abs(gain - expect) < 1e-9 * max(expect, 1e-12) + 1e-12


def test_exact_map_recovered_as_beta_vanishes(orc):
    # G = F0 E with E of full row rank (N_p > d): the fit tends to F0 as beta -> 0
    rng = np.random.default_rng(3)
    d, n_p = 16, 60
    E, G, F0 = _pairs(rng, d, n_p)
    for beta, tol in [(1e-6, 1e-6), (1e-9, 1e-9)]:
        F = orc.feedback_fit(E, G, beta)
        assert np.abs(F - F0).max() < tol * 10


def test_truncation_lemma(orc):
    rng = np.random.default_rng(4)
    d, n_p, k, beta = 28, 40, 6, 0.1
    E, G, _ = _pairs(rng, d, n_p, noise=0.3)
    F = orc.feedback_fit(E, G, beta)
    F_k, s, _, _ = orc.feedback_factors(F, k)
    np.testing.assert_allclose(s, np.linalg.svd(F, compute_uv=False), rtol=1e-11, atol=1e-13)
    # ||F - F_k||_F^2 = sum_{j>k} s_j^2 and ||(F - F_k) e|| <= s_{k+1} ||e||
    assert abs(np.sum((F - F_k) ** 2) - np.sum(s[k:] ** 2)) < 1e-10 * np.sum(s ** 2)
    for _ in range(20):
        e = rng.standard_normal(d)
        assert np.linalg.norm((F - F_k) @ e) <= s[k] * np.linalg.norm(e) * (1 + 1e-12)
    assert np.linalg.matrix_rank(F_k, tol=1e-9 * s[0]) == k


def test_credit_factors_fold_the_head(orc):
    # q_t = F_k W_u^T p_t for the head error p_t, i.e. p_t^T A~ B~ with A~ B~ = W_u F_k^T
    rng = np.random.default_rng(5)
    d, n_p, k, V = 18, 30, 5, 11
    E, G, _ = _pairs(rng, d, n_p, noise=0.2)
    Wu = rng.standard_normal((V, d))
    F_k, s, Bt, At = orc.feedback_factors(orc.feedback_fit(E, G, 0.2), k, Wu)
    assert At.shape == (V, k) and Bt.shape == (k, d)
    np.testing.assert_allclose(At @ Bt, Wu @ F_k.T, rtol=1e-10, atol=1e-11)
    p = rng.standard_normal(V)
    np.testing.assert_allclose(p @ At @ Bt, F_k @ (Wu.T @ p), rtol=1e-10, atol=1e-11)


def test_alignment_diagnostic(orc):
    rng = np.random.default_rng(6)
    d, n_p = 25, 50
    E, G, F0 = _pairs(rng, d, n_p)
    assert abs(orc.alignment(F0, E, G) - 1.0) < 1e-12          # exact map
    assert abs(orc.alignment(-F0, E, G) + 1.0) < 1e-12         # reversed map
    F = rng.standard_normal((d, d))
    assert abs(orc.alignment(3.0 * F, E, G) - orc.alignment(F, E, G)) < 1e-12  # scale invariant
    # by definition: <F E, G> / (||F E|| ||G||) written out with explicit sums
    P = F @ E
    num = sum(P[i, j] * G[i, j] for i in range(d) for j in range(n_p))
    den = np.sqrt(sum(P[i, j] ** 2 for i in range(d) for j in range(n_p))) * \
        np.sqrt(sum(G[i, j] ** 2 for i in range(d) for j in range(n_p)))
    assert abs(orc.alignment(F, E, G) - num / den) < 1e-12
