"""Pins of the oracle's paper-order head (Section S11): the top error at the hidden
width, e_t = W_u^T E_t, computed once, then the per-block coordinates V_k^T e_t.  Each
check uses a fact that holds whatever the implementation: a brute-force sum over the
classes, the invariances of the softmax error, and agreement with the folded order
(A~ = W_u V_k) computed by the oracle's separate C routines."""
from __future__ import annotations

import math

import numpy as np


def _case(rng, n=7, V=11, d=5, k=3):
    z = rng.standard_normal((n, V)) * 2.0
    y = rng.integers(0, V, n).astype(np.int32)
    Wu = rng.standard_normal((V, d))
    Vk = rng.standard_normal((d, k))
    B = rng.standard_normal((k, d))
    return z, y, Wu, Vk, B


def test_top_error_brute_force(orc):
    rng = np.random.default_rng(21)
    z, y, Wu, _, _ = _case(rng)
    w = rng.uniform(0.0, 2.0, z.shape[0])
    e = orc.top_error(z, y, Wu, w)
    n, V = z.shape
    for t in range(n):
        den = sum(math.exp(z[t, c]) for c in range(V))
        for j in range(Wu.shape[1]):
            ref = sum(w[t] * (math.exp(z[t, c]) / den - (1.0 if c == y[t] else 0.0)) * Wu[c, j] for c in range(V))
            assert abs(e[t, j] - ref) <= 1e-12 * (1 + abs(ref))


def test_top_error_invariances(orc):
    rng = np.random.default_rng(22)
    z, y, Wu, _, _ = _case(rng, n=9, V=13, d=6)
    e = orc.top_error(z, y, Wu)
    # the error row sums to zero, so one vector added to every row of W_u changes nothing
    shift = rng.standard_normal(Wu.shape[1])
    np.testing.assert_allclose(orc.top_error(z, y, Wu + shift[None, :]), e, rtol=1e-11, atol=1e-12)
    # softmax ignores a per-row logit offset
    np.testing.assert_allclose(orc.top_error(z + rng.standard_normal((z.shape[0], 1)) * 5, y, Wu), e,
                               rtol=1e-11, atol=1e-12)
    # masked positions give zero rows; weights scale rows
    w = np.ones(z.shape[0])
    w[[1, 4]] = 0.0
    w[2] = 3.0
    ew = orc.top_error(z, y, Wu, w)
    assert np.all(ew[[1, 4]] == 0.0)
    np.testing.assert_allclose(ew[2], 3.0 * e[2], rtol=1e-13)


def test_paper_order_equals_folded_order(orc):
    # F e_t through V_k^T e_t equals the folded credit factor A~ = W_u V_k applied to E_t
    rng = np.random.default_rng(23)
    z, y, Wu, Vk, B = _case(rng, n=15, V=17, d=8, k=4)
    w = rng.uniform(0.0, 2.0, z.shape[0])
    Y_p, Q_p = orc.credit_from_top_error(orc.top_error(z, y, Wu, w), Vk, B)
    Y_f, Q_f = orc.credit(orc.head_error(z, y, w), Wu @ Vk, B)
    np.testing.assert_allclose(Y_p, Y_f, rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(Q_p, Q_f, rtol=1e-11, atol=1e-12)
