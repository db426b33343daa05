"""GPU parity of the head in the paper's order (Section S11) through the C ABI: the top
error at the hidden width e_t = W_u^T E_t computed once (loca_top_error), the per-block
coordinates V_k^T e_t and ||Q||^2 (loca_credit_from_top_error), and their agreement with
the folded order (loca_error_targets with A~ = W_u V_k), against the oracle on the same
seeded inputs."""
from __future__ import annotations

import numpy as np
import pytest

from gpu_helpers import log, rel, to_dev
from paper_2608_03020_amd import inputs as gen

pytestmark = pytest.mark.gpu

TOL = 1e-5  # intermediates (e, Y, ||Q||^2)


def _inputs(n, V, d, zdt, seed, masked=0.2):
    rng = np.random.default_rng(seed)
    z = (rng.standard_normal((n, V)) * 2.0).astype(np.float32)
    y = rng.integers(0, V, n).astype(np.int32)
    w = rng.uniform(0.0, 2.0, n).astype(np.float32)
    w[rng.random(n) < masked] = 0.0
    Wu = gen.bf16_bits((rng.standard_normal((V, d)) / np.sqrt(d)).astype(np.float32))
    z_dev = gen.bf16_bits(z) if zdt == "bf16" else z
    return z_dev, y, w, Wu


@pytest.mark.parametrize("n,V,d,zdt,ld_pad", [
    (300, 1000, 64, "bf16", 0),        # ragged tokens, vocabulary chunks and one narrow column tile
    (130, 5003, 136, "f32", 5),        # ragged everything, padded logit rows (f32)
    (256, 151936, 896, "bf16", 0),     # full vocabulary at the 0.5B width
])
def test_top_error_parity(n, V, d, zdt, ld_pad):
    import torch
    import oracle
    from paper_2608_03020_amd import loca
    log(f"case top_error: n={n} V={V} d={d} logits {zdt} ld pad {ld_pad}")
    z, y, w, Wu = _inputs(n, V, d, zdt, seed=31)
    dev = "cuda"
    if ld_pad:
        zp = np.zeros((n, V + ld_pad), z.dtype)
        zp[:, :V] = z
        z_d = to_dev(zp, dev)[:, :V]
    else:
        z_d = to_dev(z, dev)
    e = torch.empty((n, d), dtype=torch.float32, device=dev)
    info = torch.full((1,), -1, dtype=torch.int32, device=dev)
    ws = loca.alloc_workspace(loca.workspace_size(loca.LOCA_OP_TOP_ERROR, 1, n, d, 1, V), dev)
    loca.loca_top_error(z_d, to_dev(y, dev), to_dev(Wu, dev), e, info, ws, w=to_dev(w, dev))
    torch.cuda.synchronize()
    assert int(info.item()) == 0
    e_ref = oracle.top_error(gen.as_f64(z, zdt), y, gen.as_f64(Wu, "bf16"), w.astype(np.float64))
    err = rel(e.double().cpu().numpy(), e_ref)
    masked = w == 0.0
    log(f"top_error n={n} V={V} d={d}: rel {err:.2e}; masked rows zero: {bool(np.all(e.cpu().numpy()[masked] == 0))}")
    assert err <= TOL
    assert np.all(e.cpu().numpy()[masked] == 0.0)


def test_top_error_bad_label_reported():
    import torch
    from paper_2608_03020_amd import loca
    n, V, d = 40, 200, 16
    z, y, w, Wu = _inputs(n, V, d, "bf16", seed=32, masked=0.0)
    y[17] = V
    y[29] = -1
    log("case top_error_bad_label: rows 17 and 29 out of range")
    e = torch.empty((n, d), dtype=torch.float32, device="cuda")
    info = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    ws = loca.alloc_workspace(loca.workspace_size(loca.LOCA_OP_TOP_ERROR, 1, n, d, 1, V), "cuda")
    loca.loca_top_error(to_dev(z), to_dev(y), to_dev(Wu), e, info, ws)
    torch.cuda.synchronize()
    assert int(info.item()) == 18


@pytest.mark.parametrize("nb,n,d,k", [(3, 200, 136, 24), (2, 129, 64, 100)])
def test_credit_from_top_error_parity(nb, n, d, k):
    import torch
    import oracle
    from paper_2608_03020_amd import loca
    log(f"case credit_from_top_error: nb={nb} n={n} d={d} k={k}")
    rng = np.random.default_rng(33)
    e = rng.standard_normal((n, d)).astype(np.float32)
    Vk = (rng.standard_normal((nb, d, k)) / np.sqrt(d)).astype(np.float32)
    B = (rng.standard_normal((nb, k, d)) / np.sqrt(k)).astype(np.float32)
    a = rng.uniform(0.0, 2.0, n).astype(np.float32)
    dev = "cuda"
    Y = torch.empty((nb, n, k), dtype=torch.float32, device=dev)
    mb = loca.new_mb(nb, dev)
    ws = loca.alloc_workspace(loca.workspace_size(loca.LOCA_OP_CREDIT_FROM_TOP_ERROR, nb, n, d, k), dev)
    loca.loca_credit_from_top_error(to_dev(e, dev), to_dev(Vk, dev), to_dev(B, dev), Y, mb, ws, a_w=to_dev(a, dev))
    torch.cuda.synchronize()
    mbh = mb.cpu().numpy()
    for b in range(nb):
        Y_ref, Q_ref = oracle.credit_from_top_error(e.astype(np.float64), Vk[b], B[b])
        q2_ref = float(np.sum(a.astype(np.float64)[:, None] * Q_ref ** 2))
        ey = rel(Y[b].double().cpu().numpy(), Y_ref)
        eq = abs(mbh[b, 0] - q2_ref) / q2_ref
        log(f"credit_from_top_error block {b}: Y {ey:.2e}, q2 {eq:.2e}")
        assert ey <= TOL and eq <= TOL


@pytest.mark.parametrize("adt", ["f32", "bf16"])
def test_paper_order_matches_folded_order(adt):
    """The same credit coordinates two ways on the GPU: the paper's order (top error once,
    then V_k^T e per block) and the folded factor A~ = W_u V_k in the error kernel (fp32 A~:
    the streaming large-vocabulary kernel; bf16 A~: one matrix-core product for all blocks,
    compared with the oracle's folded order on the same bf16 A~)."""
    import torch
    import oracle
    from paper_2608_03020_amd import loca
    nb, n, V, d, k = 3, 257, 3000, 128, 16
    log(f"case paper_vs_folded: nb={nb} n={n} V={V} d={d} k={k} A~ {adt}")
    z, y, w, Wu = _inputs(n, V, d, "f32", seed=34)
    rng = np.random.default_rng(35)
    Vk = (rng.standard_normal((nb, d, k)) / np.sqrt(d)).astype(np.float32)
    B = (rng.standard_normal((nb, k, d)) / np.sqrt(k)).astype(np.float32)
    Wu64 = gen.as_f64(Wu, "bf16")
    At = np.stack([(Wu64 @ Vk[b].astype(np.float64)).astype(np.float32) for b in range(nb)])
    if adt == "bf16":
        At = gen.bf16_bits(At)
    dev = "cuda"
    z_d, y_d, w_d = to_dev(z, dev), to_dev(y, dev), to_dev(w, dev)
    e = torch.empty((n, d), dtype=torch.float32, device=dev)
    info = torch.zeros(1, dtype=torch.int32, device=dev)
    ws = loca.alloc_workspace(max(loca.workspace_size(loca.LOCA_OP_TOP_ERROR, 1, n, d, 1, V),
                                  loca.workspace_size(loca.LOCA_OP_CREDIT_FROM_TOP_ERROR, nb, n, d, k),
                                  loca.workspace_size(loca.LOCA_OP_ERROR_TARGETS, nb, n, d, k, V)), dev)
    Yp = torch.empty((nb, n, k), dtype=torch.float32, device=dev)
    Yf = torch.empty((nb, n, k), dtype=torch.float32, device=dev)
    mbp, mbf = loca.new_mb(nb, dev), loca.new_mb(nb, dev)
    loca.loca_top_error(z_d, y_d, to_dev(Wu, dev), e, info, ws, w=w_d)
    loca.loca_credit_from_top_error(e, to_dev(Vk, dev), to_dev(B, dev), Yp, mbp, ws)
    loca.loca_error_targets(z_d, y_d, to_dev(At, dev), to_dev(B, dev), Yf, mbf, info, ws, w=w_d)
    torch.cuda.synchronize()
    assert int(info.item()) == 0
    e_ref = oracle.top_error(z.astype(np.float64), y, Wu64, w.astype(np.float64))
    E_ref = oracle.head_error(z.astype(np.float64), y, w.astype(np.float64))
    for b in range(nb):
        Y_ref, Q_ref = oracle.credit_from_top_error(e_ref, Vk[b], B[b])
        Yf_ref, Qf_ref = oracle.credit(E_ref, gen.as_f64(At[b], adt), B[b])
        ep = rel(Yp[b].double().cpu().numpy(), Y_ref)
        ef = rel(Yf[b].double().cpu().numpy(), Yf_ref)
        q2 = float(np.sum(Q_ref ** 2))
        q2f = float(np.sum(Qf_ref ** 2))
        eqp = abs(mbp[b, 0].item() - q2) / q2
        eqf = abs(mbf[b, 0].item() - q2f) / q2f
        log(f"paper_vs_folded block {b}: Y paper {ep:.2e}, Y folded {ef:.2e}, q2 paper {eqp:.2e}, folded {eqf:.2e}")
        assert max(ep, ef, eqp, eqf) <= TOL
