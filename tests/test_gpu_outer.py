"""The Jacobi outer iteration (Section S8) through the C ABI on a synthetic network of
linear residual blocks, against the oracle's outer iteration.

The network (h_l = h_{l-1} (I + F_l) + h_{l-1} W_l, logits h_L W_u^T) stands in for the
frozen backbone; its forward pass is the caller's, here float64 torch on the device for
the GPU run and numpy for the oracle, with block inputs and logits handed to the step in
float32 on both sides (fp32 mode: fp64 statistics and solve).  The credit factors are the
rank-k factors of the network's exact feedback maps, so the cross-entropy falls.  Three
steps: the adapters after each step and the losses must agree within fp32-mode
tolerance (1e-5 relative).
"""
import numpy as np
import pytest

from gpu_helpers import log, rel
from paper_2608_03020_amd import inputs as gen

pytestmark = pytest.mark.gpu


def _exact_credit(Fs, Wu, k):
    L, d = Fs.shape[0], Fs.shape[1]
    As, Bs = [], []
    for l in range(L):
        P = np.eye(d)
        for m in range(l + 1, L):
            P = P @ (np.eye(d) + Fs[m].astype(np.float64))
        U, s, Vt = np.linalg.svd(P)
        As.append(np.ascontiguousarray(Wu.astype(np.float64) @ Vt[:k].T, dtype=np.float32))
        Bs.append(np.ascontiguousarray(s[:k, None] * U[:, :k].T, dtype=np.float32))
    return As, Bs


def test_jacobi_outer_loop_matches_oracle():
    import torch
    import oracle
    from paper_2608_03020_amd.step import JacobiOuterLoop
    cfg = gen.custom_config("outer", blocks=3, d=96, n=600, micro=250, C=5, k=8, r_a=6, lambdas=(1e-2,),
                            mode="fp32", eta=0.05)
    steps = 3
    h0, Fs, Wu, y = gen.gen_linear_network(cfg)
    As, Bs = _exact_credit(Fs, Wu, cfg.k)
    log(f"case outer loop: L={cfg.blocks} d={cfg.d} n={cfg.n} micro={cfg.micro} k={cfg.k} r_a={cfg.r_a}")
    ref = oracle.jacobi_outer_loop(h0, Fs, Wu, y, [a.astype(np.float64) for a in As],
                                   [b.astype(np.float64) for b in Bs], cfg.eta, cfg.lambdas[0], cfg.r_a, steps,
                                   cfg.micro, f32_inputs=True)
    dev = "cuda"
    h0_d = torch.from_numpy(h0).to(dev, torch.float64)
    F_d = torch.from_numpy(Fs).to(dev, torch.float64)
    Wu_d = torch.from_numpy(Wu).to(dev, torch.float64)
    y_d = torch.from_numpy(y).to(dev)
    A_d = torch.from_numpy(np.stack(As)).to(dev)
    B_d = torch.from_numpy(np.stack(Bs)).to(dev)
    loop = JacobiOuterLoop(cfg, cfg.blocks, dev)

    def forward():
        lp, rp = loop.adapters()
        h, xs = h0_d, []
        for l in range(cfg.blocks):
            xs.append(h)
            h = h + h @ F_d[l] + (h @ lp[l].double()) @ rp[l].double()
        z = h @ Wu_d.T
        loss = torch.nn.functional.cross_entropy(z, y_d.long()).item()
        return torch.stack(xs).float().contiguous(), z.float().contiguous(), loss

    losses = []
    for t in range(steps):
        x_all, z, loss = forward()
        losses.append(loss)
        loop.update(x_all, z, y_d, A_d, B_d)
        torch.cuda.synchronize()
        assert np.all(loop.step.info.cpu().numpy() == 0)
        lp, rp = loop.adapters()
        errs = [rel((lp[l].double() @ rp[l].double()).cpu().numpy(), ref[t]["W"][l]) for l in range(cfg.blocks)]
        log(f"outer step {t}: loss gpu {loss:.8f} oracle {ref[t]['loss']:.8f}; adapter errors " +
            ", ".join(f"{e:.2e}" for e in errs))
        assert abs(loss - ref[t]["loss"]) <= 1e-6 * abs(ref[t]["loss"])
        assert max(errs) <= 1e-5
    _, _, loss = forward()
    losses.append(loss)
    log(f"cross-entropy over the steps: {['%.6f' % v for v in losses]}")
    assert abs(loss - ref[steps]["loss"]) <= 1e-6 * abs(ref[steps]["loss"])
    assert losses[-1] < losses[0]
