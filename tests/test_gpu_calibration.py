"""GPU parity of the Stage I calibration (Section S5) through the C ABI: the feedback
ridge fit, its rank-k truncation, the credit factors of the hot path and the
alignment diagnostic, against the oracle on the same seeded probe pairs."""
from __future__ import annotations

import numpy as np
import pytest

from gpu_helpers import log, rel, to_dev
from paper_2608_03020_amd import inputs as gen

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("d,n_p,k,nb,vocab,beta,wdt", [
    (300, 48, 8, 2, 37, 0.5, "f32"),      # ragged against the 32-row chunks
    (1024, 64, 16, 3, 200, 0.05, "bf16"),  # largest probe count, bf16 head
    (64, 5, 5, 1, 4, 1.0, "f32"),          # k = np, tiny
])
def test_feedback_fit_parity(d, n_p, k, nb, vocab, beta, wdt):
    import torch
    import oracle
    from paper_2608_03020_amd import loca
    cfg = gen.custom_config(f"calib{d}", blocks=nb, d=d, n=64, C=vocab, k=k, r_a=min(4, k))
    log(f"case feedback_fit: d={d} np={n_p} k={k} nb={nb} vocab={vocab} beta={beta} W_u {wdt}")
    E, G = gen.gen_probe_pairs(cfg, n_p, nb)
    rng = np.random.default_rng(7)
    Wu = (rng.standard_normal((vocab, d)) / np.sqrt(d)).astype(np.float32)
    if wdt == "bf16":
        Wu_bits = gen.bf16_bits(Wu)
        Wu_exact = gen.as_f64(Wu_bits, "bf16")
    else:
        Wu_bits, Wu_exact = Wu, Wu.astype(np.float64)
    dev = "cuda"
    bt = torch.empty((nb, k, d), dtype=torch.float32, device=dev)
    at = torch.empty((nb, vocab, k), dtype=torch.float32, device=dev)
    vk = torch.empty((nb, d, k), dtype=torch.float32, device=dev)
    sig = torch.empty((nb, n_p), dtype=torch.float32, device=dev)
    alpha = torch.empty(nb, dtype=torch.float64, device=dev)
    info = torch.full((nb,), -1, dtype=torch.int32, device=dev)
    ws = loca.alloc_workspace(loca.workspace_size(loca.LOCA_OP_FEEDBACK_FIT, nb, n_p, d, k), dev)
    loca.loca_feedback_fit(to_dev(E, dev), to_dev(G, dev), beta, bt, sig, alpha, info, ws, wu=to_dev(Wu_bits, dev),
                           at_out=at, vk_out=vk)
    torch.cuda.synchronize()
    assert np.all(info.cpu().numpy() == 0)
    for b in range(nb):
        F = oracle.feedback_fit(E, G[b], beta)
        F_k, s, Bt_ref, At_ref = oracle.feedback_factors(F, k, Wu_exact)
        a_ref = oracle.alignment(F_k, E, G[b])
        Bt_g = bt[b].double().cpu().numpy()
        At_g = at[b].double().cpu().numpy()
        Vk_g = vk[b].double().cpu().numpy()
        e = {"sigma": rel(sig[b].double().cpu().numpy(), s[:n_p]),
             "AB": rel(At_g @ Bt_g, At_ref @ Bt_ref),              # = W_u F_k^T, sign-free
             "BtB": rel(Bt_g.T @ Bt_g, Bt_ref.T @ Bt_ref),         # = U_k S_k^2 U_k^T
             "F_k": rel(Bt_g.T @ Vk_g.T, F_k),                      # U_k S_k V_k^T from B~ and V_k
             "alpha": abs(float(alpha[b].item()) - a_ref)}
        log(f"feedback_fit block {b}: alpha {float(alpha[b].item()):.4f} (oracle {a_ref:.4f}); " +
            ", ".join(f"{key} {v:.2e}" for key, v in e.items()))
        assert e["sigma"] <= 1e-4 and e["AB"] <= 1e-4 and e["BtB"] <= 1e-4 and e["F_k"] <= 1e-4, e
        assert e["alpha"] <= 1e-5, e


@pytest.mark.parametrize("d,n_p,k,nb,vocab,beta,wdt", [
    (700, 100, 24, 2, 64, 0.05, "bf16"),   # beyond the dual form's probe limit, ragged d
    (1024, 128, 64, 1, 100, 0.2, "f32"),   # largest probe count and rank
    (130, 65, 8, 1, 9, 1.0, "f32"),        # one probe past 64: a second chunk of one column
])
def test_feedback_fit_primal_parity(d, n_p, k, nb, vocab, beta, wdt):
    """The primal form against the oracle's primal fit (Section S5's theorem)."""
    import torch
    import oracle
    from paper_2608_03020_amd import loca
    cfg = gen.custom_config(f"calibp{d}", blocks=nb, d=d, n=64, C=vocab, k=k, r_a=4)
    log(f"case feedback_fit_primal: d={d} np={n_p} k={k} nb={nb} vocab={vocab} beta={beta} W_u {wdt}")
    E, G = gen.gen_probe_pairs(cfg, n_p, nb)
    rng = np.random.default_rng(11)
    Wu = (rng.standard_normal((vocab, d)) / np.sqrt(d)).astype(np.float32)
    if wdt == "bf16":
        Wu_bits = gen.bf16_bits(Wu)
        Wu_exact = gen.as_f64(Wu_bits, "bf16")
    else:
        Wu_bits, Wu_exact = Wu, Wu.astype(np.float64)
    dev = "cuda"
    bt = torch.empty((nb, k, d), dtype=torch.float32, device=dev)
    at = torch.empty((nb, vocab, k), dtype=torch.float32, device=dev)
    vk = torch.empty((nb, d, k), dtype=torch.float32, device=dev)
    sig = torch.empty((nb, n_p), dtype=torch.float32, device=dev)
    alpha = torch.empty(nb, dtype=torch.float64, device=dev)
    info = torch.full((nb,), -1, dtype=torch.int32, device=dev)
    ws = loca.alloc_workspace(loca.workspace_size(loca.LOCA_OP_FEEDBACK_FIT_PRIMAL, nb, n_p, d, k), dev)
    loca.loca_feedback_fit_primal(to_dev(E, dev), to_dev(G, dev), beta, bt, sig, alpha, info, ws,
                                  wu=to_dev(Wu_bits, dev), at_out=at, vk_out=vk)
    torch.cuda.synchronize()
    assert np.all(info.cpu().numpy() == 0)
    for b in range(nb):
        F = oracle.feedback_fit(E, G[b], beta, form="primal")
        F_k, s, Bt_ref, At_ref = oracle.feedback_factors(F, k, Wu_exact)
        a_ref = oracle.alignment(F_k, E, G[b])
        Bt_g = bt[b].double().cpu().numpy()
        At_g = at[b].double().cpu().numpy()
        Vk_g = vk[b].double().cpu().numpy()
        e = {"sigma": rel(sig[b].double().cpu().numpy(), s[:n_p]),
             "AB": rel(At_g @ Bt_g, At_ref @ Bt_ref),
             "BtB": rel(Bt_g.T @ Bt_g, Bt_ref.T @ Bt_ref),
             "F_k": rel(Bt_g.T @ Vk_g.T, F_k),
             "alpha": abs(float(alpha[b].item()) - a_ref)}
        log(f"feedback_fit_primal block {b}: alpha {float(alpha[b].item()):.4f} (oracle {a_ref:.4f}); " +
            ", ".join(f"{key} {v:.2e}" for key, v in e.items()))
        assert e["sigma"] <= 1e-4 and e["AB"] <= 1e-4 and e["BtB"] <= 1e-4 and e["F_k"] <= 1e-4, e
        assert e["alpha"] <= 1e-5, e


def test_feedback_fit_primal_matches_dual():
    """At 64 probes both forms serve: the fitted factors agree (the push-through identity
    of Section S5's theorem), each to rounding."""
    import torch
    from paper_2608_03020_amd import loca
    d, n_p, k, nb = 512, 64, 16, 2
    cfg = gen.custom_config("calibpd", blocks=nb, d=d, n=64, C=16, k=k, r_a=4)
    log(f"case feedback_fit primal vs dual: d={d} np={n_p} k={k} nb={nb}")
    E, G = gen.gen_probe_pairs(cfg, n_p, nb)
    dev = "cuda"
    outs = {}
    for name, op, fn in (("dual", loca.LOCA_OP_FEEDBACK_FIT, loca.loca_feedback_fit),
                         ("primal", loca.LOCA_OP_FEEDBACK_FIT_PRIMAL, loca.loca_feedback_fit_primal)):
        bt = torch.empty((nb, k, d), dtype=torch.float32, device=dev)
        vk = torch.empty((nb, d, k), dtype=torch.float32, device=dev)
        sig = torch.empty((nb, n_p), dtype=torch.float32, device=dev)
        alpha = torch.empty(nb, dtype=torch.float64, device=dev)
        info = torch.full((nb,), -1, dtype=torch.int32, device=dev)
        ws = loca.alloc_workspace(loca.workspace_size(op, nb, n_p, d, k), dev)
        fn(to_dev(E, dev), to_dev(G, dev), 0.1, bt, sig, alpha, info, ws, vk_out=vk)
        torch.cuda.synchronize()
        assert np.all(info.cpu().numpy() == 0)
        outs[name] = (bt.double().cpu().numpy(), vk.double().cpu().numpy(), sig.double().cpu().numpy(),
                      alpha.cpu().numpy())
    (bd, vd, sd, ad), (bp, vp, sp, ap) = outs["dual"], outs["primal"]
    for b in range(nb):
        e = {"F_k": rel(bp[b].T @ vp[b].T, bd[b].T @ vd[b].T), "sigma": rel(sp[b][:k], sd[b][:k]),
             "alpha": abs(ap[b] - ad[b])}
        log(f"primal vs dual block {b}: " + ", ".join(f"{key} {v:.2e}" for key, v in e.items()))
        assert e["F_k"] <= 1e-4 and e["sigma"] <= 1e-4 and e["alpha"] <= 1e-5, e


@pytest.mark.parametrize("d,n_p,k,l,q,nb,vocab,wdt", [
    (256, 600, 8, 32, 4, 2, 40, "f32"),     # np > d: a full-rank d x d map, two blocks
    (520, 1100, 16, 48, 3, 1, 64, "bf16"),  # ragged d and np (nine solve chunks, ragged tiles)
    (384, 200, 8, 24, 3, 1, 10, "f32"),     # np < d: the same path on a rank-deficient map
    (640, 900, 64, 128, 4, 1, 20, "f32"),   # the widest basis and the largest rank
])
def test_feedback_fit_large_parity(d, n_p, k, l, q, nb, vocab, wdt):
    """Subspace iteration on the primal fit (Section S5) against the oracle's dense primal fit
    and its exact rank-k SVD.  The probe gradients follow a rank-k map plus noise, so that
    sigma_k / sigma_{k+1} is large and q rounds converge far below the tolerance."""
    import torch
    import oracle
    from paper_2608_03020_amd import loca
    cfg = gen.custom_config(f"calibl{d}", blocks=nb, d=d, n=64, C=vocab, k=k, r_a=4)
    log(f"case feedback_fit_large: d={d} np={n_p} k={k} l={l} q={q} nb={nb} vocab={vocab} W_u {wdt}")
    E, G = gen.gen_probe_pairs(cfg, n_p, nb, rank=k, noise=0.3)
    omega = np.random.default_rng(5).standard_normal((d, l)).astype(np.float32)
    rng = np.random.default_rng(13)
    Wu = (rng.standard_normal((vocab, d)) / np.sqrt(d)).astype(np.float32)
    if wdt == "bf16":
        Wu_bits = gen.bf16_bits(Wu)
        Wu_exact = gen.as_f64(Wu_bits, "bf16")
    else:
        Wu_bits, Wu_exact = Wu, Wu.astype(np.float64)
    dev = "cuda"
    bt = torch.full((nb, k, d), float("nan"), dtype=torch.float32, device=dev)
    at = torch.full((nb, vocab, k), float("nan"), dtype=torch.float32, device=dev)
    vk = torch.full((nb, d, k), float("nan"), dtype=torch.float32, device=dev)
    sig = torch.full((nb, l), float("nan"), dtype=torch.float32, device=dev)
    alpha = torch.full((nb,), float("nan"), dtype=torch.float64, device=dev)
    info = torch.full((nb,), -7, dtype=torch.int32, device=dev)
    ws = loca.alloc_workspace(loca.workspace_size(loca.LOCA_OP_FEEDBACK_FIT_LARGE, nb, n_p, d, k, r_a=l), dev)
    ws.view(torch.uint8).fill_(0xFF)  # NaN patterns: every value read must have been written
    loca.loca_feedback_fit_large(to_dev(E, dev), to_dev(G, dev), to_dev(omega, dev), q, 0.1, bt, sig, alpha, info,
                                 ws, wu=to_dev(Wu_bits, dev), at_out=at, vk_out=vk)
    torch.cuda.synchronize()
    assert np.all(info.cpu().numpy() == 0), info.cpu().numpy()
    for t in (bt, at, vk, sig, alpha):
        assert not torch.isnan(t).any()
    for b in range(nb):
        F = oracle.feedback_fit(E, G[b], 0.1, form="primal")
        F_k, s, Bt_ref, At_ref = oracle.feedback_factors(F, k, Wu_exact)
        a_ref = oracle.alignment(F_k, E, G[b])
        Bt_g = bt[b].double().cpu().numpy()
        At_g = at[b].double().cpu().numpy()
        Vk_g = vk[b].double().cpu().numpy()
        e = {"sigma_k": rel(sig[b].double().cpu().numpy()[:k], s[:k]),
             "AB": rel(At_g @ Bt_g, At_ref @ Bt_ref),
             "BtB": rel(Bt_g.T @ Bt_g, Bt_ref.T @ Bt_ref),
             "F_k": rel(Bt_g.T @ Vk_g.T, F_k),
             "alpha": abs(float(alpha[b].item()) - a_ref)}
        log(f"feedback_fit_large block {b}: alpha {float(alpha[b].item()):.4f} (oracle {a_ref:.4f}); " +
            ", ".join(f"{key} {v:.2e}" for key, v in e.items()))
        assert e["sigma_k"] <= 1e-4 and e["AB"] <= 1e-4 and e["BtB"] <= 1e-4 and e["F_k"] <= 1e-4, e
        assert e["alpha"] <= 1e-5, e
        # the Ritz values beyond k are a decreasing lower bound of the singular values
        sg = sig[b].double().cpu().numpy()
        assert np.all(np.diff(sg) <= 0) and np.all(sg <= s[:l] * (1 + 1e-5))
