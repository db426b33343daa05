"""Parity at the full workload sizes, in the launch configuration bench.py times.

For each workload the whole step runs on every block exactly as the benchmark
runs it (``bench.make_inputs`` and ``bench.run_step``).  Block 0 is then checked
against the oracle end to end, on host copies of the same seeded inputs: the head
error and credit coordinates of every micro-batch (over the whole vocabulary for
the full-vocabulary workload), the last micro-batch's ||X||^2, ||Q||^2 and
eta-bar, the full S and K, the ridge solution M of every lambda (Theorem S6.1;
Section S7's Cholesky solve), and the rank-r_a truncation: singular values and
the adapter W_r (the rank-truncation lemma of Section S5).  The oracle's
statistics use a library matrix product at these widths (gram_matmul,
cross_matmul, credit_matmul; pinned against its plain loops on the CPU).
The last block is checked by sampled S entries against the oracle and by
properties that hold at any size (the solve's normwise backward error against
the GPU's S and K, the truncation against an exact SVD of the GPU's M B~).
"""
from __future__ import annotations

import os
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from gpu_helpers import log, rel  # noqa: E402

pytestmark = pytest.mark.gpu

TOL = {"bf16": 2e-3, "fp32": 1e-5}
TOL_INTER = 1e-5        # Y, ||X||^2, ||Q||^2, eta-bar
TOL_BACKWARD = 1e-5     # ||(S + lam I) M - K|| / (||S + lam I|| ||M|| + ||K||), float arithmetic


def host64(t):
    """Exact float64 host copy of a device tensor (bf16, fp32 or fp64)."""
    import torch
    return t.to(torch.float64).cpu().numpy()


def sym_from_upper(Su):
    U = np.triu(Su)
    return U + U.T - np.diag(np.diag(U))


def eckart_young(M, B, r):
    """Singular values of W = M B (M: d x k, B: k x d) and the rank-r factors
    (P, Q) with W_r = P Q^T, from QR factors and a k x k SVD."""
    Qm, Rm = np.linalg.qr(M)
    Qb, Rb = np.linalg.qr(B.T)
    U, s, Vt = np.linalg.svd(Rm @ Rb.T)
    P = Qm @ U[:, :r] * s[:r]
    Q = Qb @ Vt[:r].T
    return s, P, Q


def lowrank_diff(P1, Q1, P2, Q2):
    """||P1 Q1^T - P2 Q2^T||_F / ||P2 Q2^T||_F without forming d x d matrices."""
    def ip(Pa, Qa, Pb, Qb):
        return float(np.trace((Pa.T @ Pb) @ (Qb.T @ Qa)))
    n1, n2, x = ip(P1, Q1, P1, Q1), ip(P2, Q2, P2, Q2), ip(P1, Q1, P2, Q2)
    return float(np.sqrt(max(n1 + n2 - 2 * x, 0.0) / max(n2, 1e-300)))


def check_solve_and_truncation(cfg, step, b, Bb, tol):
    """Properties of the solve and the truncation of block b (all lambdas)."""
    nl = len(cfg.lambdas)
    S = sym_from_upper(host64(step.S[b]))
    K = host64(step.K[b])
    errs = {}
    for l, lam in enumerate(cfg.lambdas):
        M = host64(step.M[b, l])
        A_l = S + lam * np.eye(cfg.d)
        res = A_l @ M - K
        back = np.linalg.norm(res) / (np.linalg.norm(A_l) * np.linalg.norm(M) + np.linalg.norm(K))
        errs[f"backward{l}"] = float(back)
        assert back <= TOL_BACKWARD, f"block {b} lambda {lam}: backward error {back:.2e}"
        mi = b * nl + l
        s_ref, P_ref, Q_ref = eckart_young(M, Bb, cfg.r_a)
        sig = host64(step.sigma[mi])
        errs[f"sigma{l}"] = rel(sig, s_ref[:cfg.k])
        A_ad = host64(step.A_ad[mi])  # r_a x d
        B_ad = host64(step.B_ad[mi])  # d x r_a
        errs[f"Wr{l}"] = lowrank_diff(A_ad.T, B_ad, P_ref, Q_ref)
        # directions whose singular value is below the float resolution of M carry no
        # weight, their rows an orthonormal completion: every row is checked
        errs[f"orth{l}"] = float(np.abs(A_ad @ A_ad.T - np.eye(cfg.r_a)).max())
        assert errs[f"sigma{l}"] <= 1e-4 and errs[f"Wr{l}"] <= tol and errs[f"orth{l}"] <= 1e-4, errs
    return errs


def oracle_block(cfg, x_b, z, y_h, Ab, Bb):
    """The oracle's chain for one block on the exact input values: per micro-batch the
    head error, the credit coordinates, the scale normalisation and K; S; then M, the
    singular values and the rank-r_a factors for every lambda."""
    import oracle
    n_mb = cfg.n_micro
    K = np.zeros((cfg.d, cfg.k))
    rec = []
    for m in range(n_mb):
        lo, hi = cfg.micro_rows(m)
        if cfg.C <= 4096:
            E = oracle.head_error(host64(z[lo:hi]), y_h[lo:hi])
        else:
            # the full vocabulary, converted to float64 in slices of 256 tokens
            E = np.concatenate([oracle.head_error(host64(z[t0:min(hi, t0 + 256)]), y_h[t0:min(hi, t0 + 256)])
                                for t0 in range(lo, hi, 256)])
        Y, Q = oracle.credit_matmul(E, Ab, Bb)
        del E
        _, st = oracle.scaled_target(x_b[lo:hi], Q, cfg.eta)
        del Q
        K += oracle.cross_matmul(x_b[lo:hi], -st["eta_bar"] * Y)
        rec.append((Y, st))
    S = oracle.gram_matmul(x_b)
    sols = []
    for lam in cfg.lambdas:
        M, resid = oracle.ridge_solve(S, K, lam)
        _, sig, a, b = oracle.truncate_factored(M, Bb, cfg.r_a, want_dense=False)
        sols.append({"M": M, "resid": resid, "sigma": sig, "a": a, "b": b})
    return S, K, rec, sols


def run_workload(name, nb_cap=None):
    import time
    import torch
    import bench
    import oracle
    from paper_2608_03020_amd.inputs import CONFIGS
    from paper_2608_03020_amd.step import BlockStep
    cfg = CONFIGS[name]
    nb = cfg.blocks if nb_cap is None else min(cfg.blocks, nb_cap)
    log(f"[fullsize] {name}: {nb} blocks, d={cfg.d}, N={cfg.n} ({cfg.n_micro} x {cfg.micro}), C={cfg.C}, k={cfg.k}, "
        f"r_a={cfg.r_a}, lambdas={cfg.lambdas}, mode={cfg.mode}: bench inputs and one bench step")
    dev = torch.device("cuda:0")
    x_all, z, y, A, B = bench.make_inputs(cfg, nb)
    step = BlockStep(cfg, nb, dev, poison=True)
    bench.run_step(step, cfg, nb, x_all, z, y, A, B, torch.cuda.current_stream())
    torch.cuda.synchronize()
    info = step.info.cpu().numpy()
    assert np.all(info == 0), f"dev_info {info}"
    for nm_, t in (("M", step.M), ("A", step.A_ad), ("B", step.B_ad), ("sigma", step.sigma)):
        assert not bool(torch.isnan(t).any()), f"{nm_} has unwritten (NaN) entries"
    tol = TOL[cfg.mode]
    y_h = y.cpu().numpy()
    mb = step.mb.cpu().numpy()  # last micro-batch: sum_q2, sum_x2, eta_bar, n
    rng = np.random.default_rng(20260)
    nl = len(cfg.lambdas)

    # block 0: the oracle end to end
    b = 0
    t0 = time.time()
    log(f"[fullsize] {name}: oracle on block {b}")
    Ab, Bb, x_b = host64(A[b]), host64(B[b]), host64(x_all[b])
    S_ref, K_ref, rec, sols = oracle_block(cfg, x_b, z, y_h, Ab, Bb)
    errs = {}
    lo_l, hi_l = cfg.micro_rows(cfg.n_micro - 1)
    Y_last, st_last = rec[-1]
    errs["Y"] = rel(host64(step.Y[b, :hi_l - lo_l]), Y_last)
    errs["x2"] = abs(mb[b, 1] - st_last["sum_x2"]) / st_last["sum_x2"]
    errs["q2"] = abs(mb[b, 0] - st_last["sum_q2"]) / st_last["sum_q2"]
    errs["eta"] = abs(mb[b, 2] - st_last["eta_bar"]) / st_last["eta_bar"]
    errs["S"] = rel(np.triu(host64(step.S[b])), np.triu(S_ref))
    errs["K"] = rel(host64(step.K[b]), K_ref)
    for l in range(nl):
        sol = sols[l]
        mi = b * nl + l
        errs[f"resid{l}"] = sol["resid"]
        errs[f"M{l}"] = rel(host64(step.M[b, l]), sol["M"])
        kp = cfg.k
        errs[f"sigma{l}"] = rel(host64(step.sigma[mi])[:kp], sol["sigma"][:kp])
        errs[f"Wr{l}"] = lowrank_diff(host64(step.A_ad[mi]).T, host64(step.B_ad[mi]), sol["a"].T, sol["b"])
        s_r = sol["sigma"]
        errs[f"gap{l}"] = float(s_r[cfg.r_a - 1] / s_r[cfg.r_a]) if cfg.r_a < kp and s_r[cfg.r_a] > 0 else float("inf")
    log(f"[fullsize] {name} block {b} vs oracle ({time.time() - t0:.1f} s): " +
        ", ".join(f"{k} {v:.2e}" for k, v in errs.items()))
    for key in ("Y", "x2", "q2", "eta"):
        assert errs[key] <= TOL_INTER, (key, errs[key])
    for key in ["S", "K"] + [f"{q}{l}" for l in range(nl) for q in ("M", "sigma", "Wr")]:
        assert errs[key] <= tol, (key, errs[key], errs)
    del x_b, S_ref, K_ref, rec, sols

    # last block: sampled S entries against the oracle, the solve and truncation by properties
    b = nb - 1
    if b > 0:
        x_b, Bb = host64(x_all[b]), host64(B[b])
        errs = {}
        pairs = np.concatenate([
            np.sort(rng.integers(0, cfg.d, size=(256, 2)), axis=1),
            np.stack([rng.integers(0, cfg.d, 64)] * 2, axis=1)])
        S_smp = oracle.gram_entries(x_b, pairs)
        S_gpu = host64(step.S[b])[pairs[:, 0], pairs[:, 1]]
        errs["S_sampled"] = rel(S_gpu, S_smp)
        errs.update(check_solve_and_truncation(cfg, step, b, Bb, tol))
        log(f"[fullsize] {name} block {b}: " + ", ".join(f"{k} {v:.2e}" for k, v in errs.items()))
        assert errs["S_sampled"] <= tol, errs
    del x_all, step
    torch.cuda.empty_cache()


@pytest.mark.parametrize("name", ["c1", "c2", "c3", "c4", "c5"])
def test_fullsize_parity(name):
    run_workload(name)
