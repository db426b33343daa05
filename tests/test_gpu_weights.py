"""GPU parity of the weighted statistics through the C ABI: explicit nonnegative
position weights a_t in S, K and the ridge objective (Section S7's weighted form),
with the mean squares of the scale normalisation (Eq. 10) under the same weights.
Every statistics kernel path is covered, against the oracle on the same seeded
inputs, plus two identities the weighted bf16 path must meet exactly: a = 1 gives
the unweighted results bit for bit, and a = 2 doubles S and K bit for bit."""
from __future__ import annotations

import numpy as np
import pytest

from gpu_helpers import host_inputs, log, padded_rows, rel, to_dev
from paper_2608_03020_amd import inputs as gen

pytestmark = pytest.mark.gpu

CASES = {
    # name: (d, n, micro, C, k, mode)
    "dl_fused": (1024, 2600, 1300, 5, 16, "bf16"),    # direct-to-LDS Gram, cross statistic fused; ragged stages
    "dl_cross": (1024, 2300, 2300, 300, 40, "bf16"),  # cross statistic in its own launch (2k > 64); C > 64 error kernel
    "staged_128": (300, 900, 450, 5, 8, "bf16"),      # register-staged 128-wide tiles (d < 1024)
    "staged_256": (1100, 2500, 2500, 3, 8, "bf16"),   # register-staged 256-wide tiles (d % 8 != 0)
    "fp32": (200, 150, 150, 2, 4, "fp32"),            # fp64 statistics (N < d)
}
TOL = {"bf16": 2e-3, "fp32": 1e-5}


def _run(cfg, blocks, xs, zs, ys, As, Bs, a_list, dev="cuda"):
    """One pass of rows a1-a6 with statistic weights a_list[m] (None = unweighted)."""
    import torch
    from paper_2608_03020_amd.step import BlockStep
    step = BlockStep(cfg, len(blocks), dev)
    x_all = padded_rows(np.stack([np.concatenate(xb, axis=0) for xb in xs]), dev)
    z_all, y_all = to_dev(np.concatenate(zs, axis=0), dev), to_dev(np.concatenate(ys, axis=0), dev)
    A, B = to_dev(np.stack(As), dev), to_dev(np.stack(Bs), dev)
    step.reset()
    mbs = []
    for m in range(cfg.n_micro):
        lo, hi = cfg.micro_rows(m)
        a = None if a_list is None else to_dev(a_list[m], dev)
        step.micro_batch(x_all[:, lo:hi], z_all[lo:hi], y_all[lo:hi], A, B, a=a)
        mbs.append(step.mb.cpu().numpy().copy())
    step.solve(B)
    torch.cuda.synchronize()
    assert np.all(step.info.cpu().numpy() == 0), step.info.cpu().numpy()
    return step, mbs


@pytest.mark.parametrize("name", sorted(CASES))
def test_weighted_statistics_parity(name):
    import oracle
    d, n, micro, C, k, mode = CASES[name]
    cfg = gen.custom_config(f"w_{name}", blocks=2, d=d, n=n, micro=micro, C=C, k=k, r_a=min(8, k),
                            lambdas=(1e-2,), mode=mode,
                            x_dist="gauss_outlier" if mode == "fp32" else "rms_outlier")
    blocks = [0, 1]
    log(f"case weighted_stats {name}: d={d} n={n} micro={micro} C={C} k={k} mode={mode}, 20% zero weights")
    xs, zs, ys, As, Bs = host_inputs(cfg, blocks)
    a_list = [gen.gen_stat_weights(cfg, m) for m in range(cfg.n_micro)]
    step, mbs = _run(cfg, blocks, xs, zs, ys, As, Bs, a_list)
    tol = TOL[mode]
    for b in blocks:
        xf = [gen.as_f64(x, "bf16" if mode == "bf16" else "f32") for x in xs[b]]
        o = oracle.block_step(xf, [gen.as_f64(z, cfg.logit_dtype) for z in zs], ys, gen.as_f64(As[b], cfg.a_dtype),
                              np.asarray(Bs[b], np.float64), cfg.eta, cfg.lambdas, cfg.r_a,
                              a_ws=[np.asarray(a, np.float64) for a in a_list], dense_truncation=False)
        e = {}
        for m in range(cfg.n_micro):
            om = o["mb"][m]
            e[f"x2_{m}"] = abs(mbs[m][b, 1] - om["sum_x2"]) / om["sum_x2"]
            e[f"q2_{m}"] = abs(mbs[m][b, 0] - om["sum_q2"]) / om["sum_q2"]
            e[f"eta{m}"] = abs(mbs[m][b, 2] - om["eta_bar"]) / om["eta_bar"]
        iu = np.triu_indices(cfg.d)
        e["S"] = rel(step.S[b].double().cpu().numpy()[iu], o["S"][iu])
        e["K"] = rel(step.K[b].double().cpu().numpy(), o["K"])
        e["M"] = rel(step.M[b, 0].double().cpu().numpy(), o["solves"][0]["M"])
        log(f"weighted_stats {name} block {b}: " + ", ".join(f"{key} {v:.2e}" for key, v in e.items()))
        assert max(v for key, v in e.items() if key[0] in "xqe") <= 1e-5, e
        assert e["S"] <= tol and e["K"] <= tol and e["M"] <= tol, e


@pytest.mark.parametrize("name", ["dl_fused", "dl_cross", "staged_256"])
def test_weighted_statistics_exact_scalings(name):
    d, n, micro, C, k, mode = CASES[name]
    cfg = gen.custom_config(f"w_{name}", blocks=2, d=d, n=n, micro=micro, C=C, k=k, r_a=min(8, k), mode=mode)
    blocks = [0, 1]
    log(f"case weighted_stats_exact {name}: a = 1 and a = 2 against the unweighted call")
    xs, zs, ys, As, Bs = host_inputs(cfg, blocks)
    base, mb0 = _run(cfg, blocks, xs, zs, ys, As, Bs, None)
    S0, K0 = base.S.cpu().numpy(), base.K.cpu().numpy()
    del base
    ones = [np.ones(cfg.micro_rows(m)[1] - cfg.micro_rows(m)[0], np.float32) for m in range(cfg.n_micro)]
    one, mb1 = _run(cfg, blocks, xs, zs, ys, As, Bs, ones)
    iu = np.triu_indices(cfg.d)
    for b in blocks:
        assert np.array_equal(one.S[b].cpu().numpy()[iu], S0[b][iu]), "a = 1 must reproduce the unweighted S"
        assert np.array_equal(one.K[b].cpu().numpy(), K0[b]), "a = 1 must reproduce the unweighted K"
    assert np.array_equal(mb1[-1], mb0[-1])
    del one
    twos = [2.0 * a for a in ones]
    two, mb2 = _run(cfg, blocks, xs, zs, ys, As, Bs, twos)
    for b in blocks:
        assert np.array_equal(two.S[b].cpu().numpy()[iu], 2.0 * S0[b][iu]), "a = 2 must double S exactly"
        assert np.array_equal(two.K[b].cpu().numpy(), 2.0 * K0[b]), "a = 2 must double K exactly"
        # the mean squares double together, so eta_bar is unchanged
        assert mb2[-1][b, 2] == mb0[-1][b, 2] or abs(mb2[-1][b, 2] / mb0[-1][b, 2] - 1) < 1e-15
    log(f"weighted_stats_exact {name}: bitwise identities hold")
