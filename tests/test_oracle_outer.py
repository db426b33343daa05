"""Pins of the oracle's outer iteration (Section S8, Jacobi schedule) on a synthetic
network of linear residual blocks.

* eta = 0 asks for no displacement: every adapter stays zero and the loss is that of
  the frozen network at every step.
* With the exact feedback map of the linear network (the Jacobian of its output with
  respect to each block's hidden state, truncated to rank k from its SVD: the rank-k map
  of Section S5 built from exact gradients) and a small eta, one Jacobi step lowers the
  cross-entropy: to first order each block's realised change is a projected gradient
  step.  A flipped sign or a transposed map raises it.
* A Jacobi step solves every block from the same forward pass: the first step's
  adapters equal the single-block solves on the frozen network's block inputs.
"""
import numpy as np

from paper_2608_03020_amd import inputs as gen


def _exact_credit(Fs, Wu, k, transpose=False):
    """Rank-k factors of the exact feedback maps of the linear network: the row
    displacement of h_l that the top error asks for is e P_l^T with P_l = prod_{m>l}
    (I + F_m), so F_l = P_l (column form) and A~ = W_u V_k, B~ = S_k U_k^T."""
    L, d = Fs.shape[0], Fs.shape[1]
    As, Bs = [], []
    for l in range(L):
        P = np.eye(d)
        for m in range(l + 1, L):
            P = P @ (np.eye(d) + Fs[m].astype(np.float64))
        U, s, Vt = np.linalg.svd(P.T if transpose else P)
        As.append(Wu.astype(np.float64) @ Vt[:k].T)
        Bs.append(s[:k, None] * U[:, :k].T)
    return As, Bs


def _net(k=None):
    cfg = gen.custom_config("lin", blocks=3, d=40, n=500, C=5, k=k or 40, r_a=40, lambdas=(1e-3,), mode="fp32")
    h0, Fs, Wu, y = gen.gen_linear_network(cfg)
    return cfg, h0, Fs, Wu, y


def test_zero_eta_keeps_the_frozen_network(orc):
    cfg, h0, Fs, Wu, y = _net(k=8)
    As, Bs = _exact_credit(Fs, Wu, 8)
    hist = orc.jacobi_outer_loop(h0, Fs, Wu, y, As, Bs, 0.0, 1e-2, 4, 2, 200)
    for h in hist[:-1]:
        assert all(np.all(W == 0.0) for W in h["W"])
    assert len({round(h["loss"], 14) for h in hist}) == 1


def test_exact_credit_step_lowers_the_loss(orc):
    cfg, h0, Fs, Wu, y = _net()
    As, Bs = _exact_credit(Fs, Wu, cfg.d)
    hist = orc.jacobi_outer_loop(h0, Fs, Wu, y, As, Bs, 0.01, 1e-3, cfg.d, 1, 250)
    assert hist[1]["loss"] < hist[0]["loss"] - 1e-4
    # the same step with the feedback map's sign flipped raises the loss
    hist_f = orc.jacobi_outer_loop(h0, Fs, Wu, y, As, [-B for B in Bs], 0.01, 1e-3, cfg.d, 1, 250)
    assert hist_f[1]["loss"] > hist_f[0]["loss"] + 1e-4
    # the transposed map F_l^T (U_k and V_k exchanged) descends less than the exact one
    At, Bt = _exact_credit(Fs, Wu, cfg.d, transpose=True)
    hist_t = orc.jacobi_outer_loop(h0, Fs, Wu, y, At, Bt, 0.01, 1e-3, cfg.d, 1, 250)
    assert hist_t[1]["loss"] > hist[1]["loss"]


def test_first_jacobi_step_is_the_single_block_solves(orc):
    cfg, h0, Fs, Wu, y = _net(k=8)
    As, Bs = _exact_credit(Fs, Wu, 8)
    hist = orc.jacobi_outer_loop(h0, Fs, Wu, y, As, Bs, 0.02, 1e-2, 4, 1, 200)
    xs, z = orc.linear_blocks_forward(h0, Fs, [None] * 3, Wu)
    rows = [(0, 200), (200, 400), (400, 500)]
    for l in range(3):
        o = orc.block_step([xs[l][lo:hi] for lo, hi in rows], [z[lo:hi] for lo, hi in rows],
                           [y[lo:hi] for lo, hi in rows], As[l], Bs[l], 0.02, (1e-2,), 4)
        np.testing.assert_allclose(hist[0]["W"][l], o["solves"][0]["W_r"], rtol=1e-9, atol=1e-14)
