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


def test_fused_head_brute_force(orc):
    # from hidden states: z_t = W_u h_t by explicit sums, softmax by explicit exponentials
    rng = np.random.default_rng(24)
    n, V, d, c = 5, 9, 4, 3
    h = rng.standard_normal((n, d))
    Wu = rng.standard_normal((V, d))
    Vm = rng.standard_normal((V, c))
    y = rng.integers(0, V, n).astype(np.int32)
    w = rng.uniform(0.0, 2.0, n)
    out = orc.fused_head(h, Wu, y, Vm, w)
    for t in range(n):
        z = [sum(Wu[v, j] * h[t, j] for j in range(d)) for v in range(V)]
        den = sum(math.exp(zv) for zv in z)
        for j in range(c):
            ref = w[t] * sum((math.exp(z[v]) / den - (1.0 if v == y[t] else 0.0)) * Vm[v, j] for v in range(V))
            assert abs(out[t, j] - ref) <= 1e-12 * (1 + abs(ref))


def test_fused_head_invariances(orc):
    rng = np.random.default_rng(25)
    n, V, d, c = 8, 12, 6, 5
    h = rng.standard_normal((n, d)) * 2.0
    Wu = rng.standard_normal((V, d))
    Vm = rng.standard_normal((V, c))
    y = rng.integers(0, V, n).astype(np.int32)
    out = orc.fused_head(h, Wu, y, Vm)
    # each error row sums to zero: a vector added to every row of Vm changes nothing
    np.testing.assert_allclose(orc.fused_head(h, Wu, y, Vm + rng.standard_normal(c)[None, :]), out,
                               rtol=1e-11, atol=1e-12)
    # a hidden direction orthogonal to every head row leaves the logits unchanged
    Vs, ds = 4, 7
    Ws = rng.standard_normal((Vs, ds))
    hs = rng.standard_normal((n, ds))
    ys = rng.integers(0, Vs, n).astype(np.int32)
    Vms = rng.standard_normal((Vs, c))
    q, _ = np.linalg.qr(np.concatenate([Ws.T, rng.standard_normal((ds, 1))], axis=1))
    u = q[:, Vs]
    assert np.abs(Ws @ u).max() < 1e-12
    np.testing.assert_allclose(orc.fused_head(hs + 3.0 * u[None, :], Ws, ys, Vms), orc.fused_head(hs, Ws, ys, Vms),
                               rtol=1e-11, atol=1e-12)
    # Vm = W_u is the paper-order top error of the logits h W_u^T
    np.testing.assert_allclose(orc.fused_head(h, Wu, y, Wu), orc.top_error(h @ Wu.T, y, Wu), rtol=1e-12,
                               atol=1e-13)
