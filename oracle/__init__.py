"""float64 oracle for the LoCA per-block adaptation step -- TEST INFRASTRUCTURE.

Only the test suite, the package's smoke check and the benchmark's CPU-baseline
leg import this module.  It wraps the plain-C routines of ``loca_oracle.c``
(built by ``oracle/build.py``) with numpy marshalling, and composes them into
the steps of one block solve in the paper's order (Section S13's outer
iteration, steps 2-5):

  1. head error E_t = w_t (softmax(z_t) - onehot(y_t))         (Lemma S3.1)
  2. feedback Y = E A~, Q = Y B~ ; per mini-batch eta_bar and the displacement
     T = -eta_bar Q                                               (Eq. 10, S8)
  3. streaming statistics S += X^T X, Z += X^T T (dense)          (Eq. 9, S7)
  4. ridge solve (S + lam I) W = S W_prev + Z by Cholesky          (Thm S6.1, S7)
  5. Eckart-Young truncation of W to rank r_a                      (Lemma S5.2)
plus the paper-literal projected form with a random A_l            (Eqs. 6-9)
and the one-time Stage I calibration that produces A~, B~: the feedback ridge
fit, its rank-k truncation and the alignment diagnostic           (Section S5),
and the head in the paper's order: the top error e_t = W_u^T E_t once, then
V_k^T e_t per block                                               (Section S11),
and the LM head from the final hidden states (logits z = W_u h_t)  (Eq. 4)

It shares no code with the HIP path and never imports it.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, List, Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.environ.get("LOCA_ORACLE_LIB", os.path.join(_HERE, "liblocaoracle.so"))
_lib = None

_D = ctypes.POINTER(ctypes.c_double)
_I64 = ctypes.c_int64


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            from .build import build_oracle
            build_oracle()
        _lib = ctypes.CDLL(_LIB_PATH)
        for name in ("loca_oracle_credit", "loca_oracle_scaled_target", "loca_oracle_gram_acc",
                     "loca_oracle_cross_acc", "loca_oracle_gram_entries", "loca_oracle_cholesky_solve",
                     "loca_oracle_qr", "loca_oracle_projected_acc"):
            getattr(_lib, name).restype = None
    return _lib


def _p(a: Optional[np.ndarray]):
    if a is None:
        return None
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(ctypes.c_void_p)


def _f64(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float64)


# ----------------------------------------------------------------- primitives


def head_error(z, y, w=None) -> np.ndarray:
    z = _f64(z)
    n, C = z.shape
    y = np.ascontiguousarray(y, dtype=np.int32)
    E = np.empty((n, C), np.float64)
    w64 = None if w is None else _f64(w)
    rc = _load().loca_oracle_head_error(_I64(n), _I64(C), _p(z), _p(y), _p(w64), _p(E))
    if rc != 0:
        raise ValueError(f"label out of range at row {-rc - 1}")
    return E


def credit(E, A, B, want_q=True):
    E, A, B = _f64(E), _f64(A), _f64(B)
    n, C = E.shape
    k, d = B.shape
    assert A.shape == (C, k)
    Y = np.empty((n, k), np.float64)
    Q = np.empty((n, d), np.float64) if want_q else None
    _load().loca_oracle_credit(_I64(n), _I64(C), _I64(k), _I64(d), _p(E), _p(A), _p(B), _p(Y), _p(Q))
    return Y, Q


def _weights(a, n):
    if a is None:
        return None
    a = _f64(a).reshape(-1)
    assert a.shape == (n,)
    return a


def scaled_target(X, Q, eta, a=None):
    """eta_bar and T = -eta_bar Q (Eq. 10); `a` are position weights (None = 1)."""
    X, Q = _f64(X), _f64(Q)
    n, d = X.shape
    T = np.empty((n, d), np.float64)
    info = np.empty(3, np.float64)
    _load().loca_oracle_scaled_target(_I64(n), _I64(d), _p(X), _p(Q), _p(_weights(a, n)), ctypes.c_double(eta),
                                      _p(T), _p(info))
    return T, {"sum_x2": info[0], "sum_q2": info[1], "eta_bar": info[2]}


def gram_acc(X, S=None, a=None):
    """S += sum_t a_t x_t x_t^T (Eq. 9; Section S7's weighted statistics)."""
    X = _f64(X)
    n, d = X.shape
    S = np.zeros((d, d), np.float64) if S is None else S
    _load().loca_oracle_gram_acc(_I64(n), _I64(d), _p(X), _p(_weights(a, n)), _p(S))
    return S


def cross_acc(X, T, Z=None, a=None):
    """Z += sum_t a_t x_t T_t^T (Eq. 9; Section S7's weighted statistics)."""
    X, T = _f64(X), _f64(T)
    n, d = X.shape
    m = T.shape[1]
    Z = np.zeros((d, m), np.float64) if Z is None else Z
    _load().loca_oracle_cross_acc(_I64(n), _I64(d), _I64(m), _p(X), _p(_weights(a, n)), _p(T), _p(Z))
    return Z


def gram_matmul(X, a=None):
    """The same Gram as gram_acc, S = sum_t a_t x_t x_t^T (Eq. 9; Section S7's weights),
    with a library matrix product as its one step: fast enough for the full workload
    widths (d up to 5120 over 65536 tokens), where the plain loops would take hours."""
    X = _f64(X)
    if a is None:
        return X.T @ X
    return X.T @ (X * _weights(a, X.shape[0])[:, None])


def cross_matmul(X, T, a=None):
    """The same cross statistic as cross_acc, sum_t a_t x_t T_t^T (Eq. 9), as one library
    matrix product."""
    X, T = _f64(X), _f64(T)
    if a is None:
        return X.T @ T
    return X.T @ (T * _weights(a, X.shape[0])[:, None])


def credit_matmul(E, A, B=None):
    """The tokenwise feedback of `credit` (Y = E A~, Q = Y B~; Sections S3, S11) with library
    matrix products, for a full vocabulary where E A~ has n * V * k terms."""
    Y = _f64(E) @ _f64(A)
    return Y, (None if B is None else Y @ _f64(B))


def gram_entries(X, pairs) -> np.ndarray:
    X = _f64(X)
    n, d = X.shape
    ij = np.ascontiguousarray(pairs, dtype=np.int64).reshape(-1, 2)
    out = np.empty(ij.shape[0], np.float64)
    _load().loca_oracle_gram_entries(_I64(n), _I64(d), _p(X), _I64(ij.shape[0]), _p(ij), _p(out))
    return out


def cholesky(A) -> np.ndarray:
    L = _f64(A).copy()
    info = _load().loca_oracle_cholesky(_I64(L.shape[0]), _p(L))
    if info != 0:
        raise np.linalg.LinAlgError(f"not positive definite at pivot {info}")
    return L


def ridge_solve(S, RHS, lam):
    S, RHS = _f64(S), _f64(RHS)
    d = S.shape[0]
    m = RHS.shape[1]
    W = np.empty((d, m), np.float64)
    resid = ctypes.c_double(0.0)
    info = _load().loca_oracle_ridge_solve(_I64(d), _I64(m), _p(S), _p(RHS), ctypes.c_double(lam), _p(W),
                                           ctypes.byref(resid))
    if info != 0:
        raise np.linalg.LinAlgError(f"ridge system not positive definite (pivot {info})")
    return W, resid.value


def svd(A):
    A = _f64(A)
    rows, cols = A.shape
    assert rows >= cols
    U = np.empty((rows, cols), np.float64)
    s = np.empty(cols, np.float64)
    V = np.empty((cols, cols), np.float64)
    _load().loca_oracle_svd(_I64(rows), _I64(cols), _p(A), _p(U), _p(s), _p(V))
    return U, s, V


def qr(A):
    A = _f64(A)
    rows, cols = A.shape
    Q = np.empty((rows, cols), np.float64)
    R = np.empty((cols, cols), np.float64)
    _load().loca_oracle_qr(_I64(rows), _I64(cols), _p(A), _p(Q), _p(R))
    return Q, R


def truncate_dense(W, r):
    W = _f64(W)
    d = W.shape[0]
    Wr = np.empty((d, d), np.float64)
    sig = np.empty(d, np.float64)
    _load().loca_oracle_truncate_dense(_I64(d), _p(W), _I64(r), _p(Wr), _p(sig))
    return Wr, sig


def truncate_factored(M, R, r, want_dense=True):
    M, R = _f64(M), _f64(R)
    d, kp = M.shape
    assert R.shape == (kp, d) and kp <= d
    Wr = np.empty((d, d), np.float64) if want_dense else None
    sig = np.empty(kp, np.float64)
    a = np.empty((r, d), np.float64)
    b = np.empty((d, r), np.float64)
    _load().loca_oracle_truncate_factored(_I64(d), _I64(kp), _p(M), _p(R), _I64(r), _p(Wr), _p(sig), _p(a), _p(b))
    return Wr, sig, a, b


def realization_error(X, T, W, W_prev=None, a=None, want_e=False):
    """Realisation error of a fitted adapter (Section S6): the fit realises the
    displacement X (W - W_prev) (token-major: row n is (W - W_prev)^T x_n, the paper's
    (B* - B^(t)) p_n) where the target asked for T (rows T_n, the paper's -s q), and
        E_fit = X (W - W_prev) - T      (the data residual B* P - R),
    formed densely by its definition (the product X (W - W_prev) by a library matmul).
    With position weights `a` (Section S7) the squared norms are weighted.  Returns
    {"fit2": sum_n a_n ||E_fit,n||^2, "tar2": sum_n a_n ||T_n||^2, "w2": ||W||_F^2}
    (and E_fit itself with want_e)."""
    X, T, W = _f64(X), _f64(T), _f64(W)
    D = W if W_prev is None else W - _f64(W_prev)
    E = X @ D - T
    wa = np.ones(X.shape[0]) if a is None else _weights(a, X.shape[0])
    out = {"fit2": float(np.sum(wa[:, None] * E * E)), "tar2": float(np.sum(wa[:, None] * T * T)),
           "w2": float(np.sum(W * W))}
    if want_e:
        out["E"] = E
    return out


def projected_acc(X, T, Aproj, Bcur=None, G=None, Cst=None, a=None):
    X, T, Aproj = _f64(X), _f64(T), _f64(Aproj)
    n, d = X.shape
    r = Aproj.shape[0]
    G = np.zeros((r, r), np.float64) if G is None else G
    Cst = np.zeros((d, r), np.float64) if Cst is None else Cst
    Bc = None if Bcur is None else _f64(Bcur)
    _load().loca_oracle_projected_acc(_I64(n), _I64(d), _I64(r), _p(X), _p(T), _p(Aproj), _p(Bc),
                                      _p(_weights(a, n)), _p(G), _p(Cst))
    return G, Cst


def projected_solve(G, Cst, lam):
    G, Cst = _f64(G), _f64(Cst)
    d, r = Cst.shape
    Bs = np.empty((d, r), np.float64)
    resid = ctypes.c_double(0.0)
    info = _load().loca_oracle_projected_solve(_I64(d), _I64(r), _p(G), _p(Cst), ctypes.c_double(lam), _p(Bs),
                                               ctypes.byref(resid))
    if info != 0:
        raise np.linalg.LinAlgError(f"projected system not positive definite (pivot {info})")
    return Bs, resid.value


# ----------------------------------------------------------------- one block


# ---------------------------------------------------------------- Stage I feedback calibration


def feedback_fit(E, G, beta, form="dual"):
    """The feedback ridge fit of Stage I (Section S5, Eq. 5 and the theorem on its
    solution): F_hat = argmin_F ||F E - G||_F^2 + beta ||F||_F^2 for probe columns
    E (top errors) and G (exact block gradients), both d x N_p.
      dual:   F_hat = G (E^T E + beta I)^{-1} E^T   (a system in N_p unknowns)
      primal: F_hat = G E^T (E E^T + beta I)^{-1}   (a system in d unknowns)
    Both are linear solves (Cholesky), never explicit inverses."""
    E, G = _f64(E), _f64(G)
    if form == "dual":
        Z, _ = ridge_solve(E.T @ E, np.ascontiguousarray(E.T), beta)   # (E^T E + beta I) Z = E^T
        return G @ Z
    Ft, _ = ridge_solve(E @ E.T, E @ G.T, beta)                         # (E E^T + beta I) F^T = E G^T
    return np.ascontiguousarray(Ft.T)


def feedback_factors(F_hat, k, Wu=None):
    """Rank-k truncation F = U_k S_k V_k^T of the fitted map (Section S5, Eq. 5 and the
    rank-truncation lemma) and the credit factors the hot path takes with W_u^T folded
    into the first: B~ = S_k U_k^T (k x d), A~ = W_u V_k (rows of W_u: vocabulary).
    Returns F_k, all singular values, B~, A~ (None without W_u)."""
    U, s, V = svd(F_hat)
    F_k = (U[:, :k] * s[:k]) @ V[:, :k].T
    Bt = s[:k, None] * U[:, :k].T
    At = None if Wu is None else _f64(Wu) @ V[:, :k]
    return F_k, s, Bt, At


def alignment(F, E, G):
    """Alignment diagnostic of Section S5: the cosine between the stacked prediction
    F E and the exact probe gradients G (Frobenius inner product)."""
    P = _f64(F) @ _f64(E)
    G = _f64(G)
    return float(np.sum(P * G) / (np.linalg.norm(P) * np.linalg.norm(G)))


def top_error(z, y, Wu, w=None):
    """Top-layer error at the hidden width, e_t = W_u^T (softmax(z_t) - onehot(y_t)) scaled
    by the loss weight (the error of the target equation with Lemma S3.1's head error):
    the head applied once per top error and shared by all blocks (Section S11's cost
    order).  z (n x V), Wu (V x d) -> e (n x d); the product is a library matmul."""
    return head_error(z, y, w) @ _f64(Wu)


def fused_head(h, Wu, y, Vm, w=None):
    """The head error applied to a right operand, starting from the final hidden states
    ("Local Targets", Eq. 4, with Lemma S3.1's head error): logits z_t = W_u h_t (a library
    matmul), E_t = w_t (softmax(z_t) - onehot(y_t)), and out = E Vm.  Vm = W_u gives the top
    error of the paper's order (Section S11); Vm = W_u V_k gives a block's coordinates."""
    return head_error(_f64(h) @ _f64(Wu).T, y, w) @ _f64(Vm)


def credit_from_top_error(e, Vk, B):
    """The rank-k feedback applied to top errors in the paper's order, F e = U_k (S_k (V_k^T e))
    (Section S11): Y = e V_k (the coordinates V_k^T e_t as rows) and Q = Y B~, B~ = S_k U_k^T."""
    Y = _f64(e) @ _f64(Vk)
    return Y, Y @ _f64(B)


def block_step(xs: Sequence[np.ndarray], zs: Sequence[np.ndarray], ys: Sequence[np.ndarray],
               A, B, eta: float, lambdas: Sequence[float], r_a: int,
               ws: Optional[Sequence[np.ndarray]] = None, W_prev=None,
               Aproj=None, Bproj_cur=None, dense_truncation: Optional[bool] = None,
               want_dense=True, a_ws: Optional[Sequence[np.ndarray]] = None) -> Dict:
    """All steps of one block over its mini-batches, in the paper's order.

    xs[m] (n_m x d), zs[m] (n_m x C), ys[m] (n_m) are float64-exact inputs of
    mini-batch m; A (C x k), B (k x d) the credit factors.  W_prev (d x d) is the
    current adapter in token-major form (None = frozen model).  Aproj (r_a x d),
    when given, adds the paper-literal projected solve with current adapter
    Bproj_cur (d x r_a, None = 0).  ws[m] are the loss weights of mini-batch m
    (Lemma S3.1), a_ws[m] its statistic weights (Section S7; None = 1).
    """
    d = B.shape[1]
    S = np.zeros((d, d), np.float64)
    Z = np.zeros((d, d), np.float64)
    K = np.zeros((d, B.shape[0]), np.float64)
    G = Cst = None
    if Aproj is not None:
        G = np.zeros((Aproj.shape[0], Aproj.shape[0]), np.float64)
        Cst = np.zeros((d, Aproj.shape[0]), np.float64)
    mbs: List[Dict] = []
    Ys, Ts, Es = [], [], []
    for m, (X, z, y) in enumerate(zip(xs, zs, ys)):
        E = head_error(z, y, None if ws is None else ws[m])
        Y, Q = credit(E, A, B)
        a = None if a_ws is None else a_ws[m]
        T, info = scaled_target(X, Q, eta, a)
        gram_acc(X, S, a)
        cross_acc(X, T, Z, a)
        cross_acc(X, -info["eta_bar"] * Y, K, a)
        if Aproj is not None:
            projected_acc(X, T, Aproj, Bproj_cur, G, Cst, a)
        mbs.append(info)
        Es.append(E)
        Ys.append(Y)
        Ts.append(T)
    out = {"S": S, "Z": Z, "K": K, "mb": mbs, "E": Es, "Y": Ys, "T": Ts, "solves": []}
    if dense_truncation is None:
        dense_truncation = d <= 256
    for lam in lambdas:
        RHS = Z.copy() if W_prev is None else S @ W_prev + Z
        W, resid = ridge_solve(S, RHS, lam)
        # factored form of the same solve: W = M [B~] (W_prev = None)
        sol = {"lam": lam, "W": W, "resid": resid}
        if W_prev is None:
            M, _ = ridge_solve(S, K, lam)
            sol["M"] = M
            if dense_truncation:
                Wr, sig = truncate_dense(W, r_a)
            else:
                Wr, sig, _, _ = truncate_factored(M, _f64(B), r_a, want_dense=want_dense)
            sol["W_r"] = Wr
            sol["sigma"] = sig
        if Aproj is not None:
            Bs, presid = projected_solve(G, Cst, lam)
            sol["B_proj"] = Bs
            sol["proj_resid"] = presid
        out["solves"].append(sol)
    if Aproj is not None:
        out["G_proj"] = G
        out["C_proj"] = Cst
    return out


# ---------------------------------------------------------------- outer iteration (Section S8)


def linear_blocks_forward(h0, Fs, Ws, Wu):
    """Forward pass of a synthetic network of L linear residual blocks (the frozen backbone
    stand-in for the outer iteration): h_l = h_{l-1} (I + F_l) + h_{l-1} W_l, token-major,
    where h_{l-1} (I + F_l) is the frozen block output and h_{l-1} W_l the adapter's
    contribution (Eq. 1 in row form, W_l = (B_l A_l)^T); logits z = h_L W_u^T.  Returns the
    block inputs [h_0 .. h_{L-1}] and z.  The products are library matmuls."""
    h = _f64(h0)
    xs = []
    for F, W in zip(Fs, Ws):
        xs.append(h)
        h = h + h @ _f64(F) + (0.0 if W is None else h @ _f64(W))
    return xs, h @ _f64(Wu).T


def cross_entropy(z, y):
    """Mean cross-entropy of logits z (n x C) against labels y."""
    z = _f64(z)
    m = z.max(axis=1, keepdims=True)
    lse = m[:, 0] + np.log(np.exp(z - m).sum(axis=1))
    return float(np.mean(lse - z[np.arange(z.shape[0]), np.asarray(y)]))


def jacobi_outer_loop(h0, Fs, Wu, y, As, Bs, eta, lam, r_a, steps, micro, f32_inputs=False):
    """The outer iteration of Section S8 with the Jacobi schedule on the synthetic linear
    network: at step t one shared forward pass with the current adapters W^(t) gives every
    block's inputs and the head error; each block then solves its ridge problem with the
    residual target of Eq. 6 (current adapter W_prev = W^(t)_l, Theorem S6.1) from the
    statistics of all micro-batches of `micro` rows, and its solution is truncated to rank
    r_a (the adapter's rank); all blocks are updated at once.  Returns per step the CE of
    the forward pass it started from and the adapters after it.  With f32_inputs the block
    inputs and logits of every forward pass are rounded to float32 before the step (the
    values a float32 caller passes)."""
    L = len(Fs)
    d = _f64(h0).shape[1]
    W = [np.zeros((d, d)) for _ in range(L)]
    n = _f64(h0).shape[0]
    rows = [(lo, min(n, lo + micro)) for lo in range(0, n, micro)]
    hist = []
    for _ in range(steps):
        xs, z = linear_blocks_forward(h0, Fs, W, Wu)
        loss = cross_entropy(z, y)
        if f32_inputs:
            xs = [x.astype(np.float32).astype(np.float64) for x in xs]
            z = z.astype(np.float32).astype(np.float64)
        Wn = []
        for l in range(L):
            res = block_step([xs[l][lo:hi] for lo, hi in rows], [z[lo:hi] for lo, hi in rows],
                             [np.asarray(y)[lo:hi] for lo, hi in rows], As[l], Bs[l], eta, (lam,), r_a,
                             W_prev=W[l], dense_truncation=False)
            Wr, _ = truncate_dense(res["solves"][0]["W"], r_a)
            Wn.append(Wr)
        W = Wn
        hist.append({"loss": loss, "W": [w.copy() for w in W]})
    xs, z = linear_blocks_forward(h0, Fs, W, Wu)
    hist.append({"loss": cross_entropy(z, y), "W": None})
    return hist

