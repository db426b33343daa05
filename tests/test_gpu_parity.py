"""Parity of the HIP path (through the C ABI) with the float64 oracle.

Tolerances (relative Frobenius error): statistics S and Z = X^T T, the dense
ridge solution and the rank-r_a adapter W_r within 2e-3 in bf16 mode and 1e-5
in fp32 mode; intermediates (credit coordinates Y, eta_bar) within 1e-5.
Sizes span several tiles with ragged edges in d and in the token count.
"""
import numpy as np
import pytest

from gpu_helpers import host_inputs, log, padded_rows, rel, run_gpu, run_oracle, to_dev
from paper_2608_03020_amd import inputs as gen

pytestmark = pytest.mark.gpu

TOL = {"bf16": 2e-3, "fp32": 1e-5}


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_03020_amd import loca
    loca.load()


def _compare(cfg, g, o, b, label):
    tol = TOL[cfg.mode]
    d = cfg.d
    iu = np.triu_indices(d)
    e = {}
    e["S"] = rel(g["S"][b][iu], o["S"][iu])
    e["K"] = rel(g["K"][b], o["K"])
    for m in range(cfg.n_micro):
        e[f"Y{m}"] = rel(g["Y"][m][b], o["Y"][m])
        e[f"eta{m}"] = abs(g["mb"][m]["eta_bar"][b] - o["mb"][m]["eta_bar"]) / max(o["mb"][m]["eta_bar"], 1e-300)
        e[f"x2_{m}"] = abs(g["mb"][m]["sum_x2"][b] - o["mb"][m]["sum_x2"]) / o["mb"][m]["sum_x2"]
        e[f"q2_{m}"] = abs(g["mb"][m]["sum_q2"][b] - o["mb"][m]["sum_q2"]) / max(o["mb"][m]["sum_q2"], 1e-300)
    nl = len(cfg.lambdas)
    for l, sol in enumerate(o["solves"]):
        e[f"M{l}"] = rel(g["M"][b, l], sol["M"])
        if "W_r" in g:
            e[f"Wr{l}"] = rel(g["W_r"][b * nl + l], sol["W_r"])
        kk = min(cfg.r_a + 1, cfg.k)
        e[f"sig{l}"] = rel(g["sigma"][b * nl + l][:kk], sol["sigma"][:kk])
    log(label, {k: f"{v:.2e}" for k, v in e.items()})
    assert e["S"] <= tol and e["K"] <= tol
    for m in range(cfg.n_micro):
        assert e[f"Y{m}"] <= 1e-5 and e[f"eta{m}"] <= 1e-5 and e[f"x2_{m}"] <= 1e-5 and e[f"q2_{m}"] <= 1e-5
    for l in range(nl):
        assert e[f"M{l}"] <= tol
        if "W_r" in g:
            assert e[f"Wr{l}"] <= tol
        assert e[f"sig{l}"] <= tol
    return e


CASES = {
    # ragged d on 128-wide tiles, two micro-batches (640 + 360 rows), two blocks, two lambdas
    "bf16_d600": gen.custom_config("t1", blocks=2, d=600, n=1000, micro=640, C=5, k=16, r_a=4, lambdas=(1e-2, 1.0)),
    # ragged d on 256-wide tiles, three micro-batches with a ragged last one.  bf16 mode keeps fp32
    # statistics, which needs N > d: with N < d rounding in S leaks into the null space of X and is
    # amplified by 1/lambda (fp32 mode, with fp64 statistics, covers N < d).
    "bf16_d1100": gen.custom_config("t2", blocks=1, d=1100, n=2300, micro=1000, C=3, k=32, r_a=8),
    # d % 8 == 0 and d >= 1024: the direct-to-LDS Gram kernel; ragged against 256-wide tiles and
    # against the 32-token stages (1400 = 43 x 32 + 24), two blocks
    "bf16_d1040_direct": gen.custom_config("t10", blocks=2, d=1040, n=2400, micro=1400, C=4, k=16, r_a=4),
    # cross statistic inside the Gram launch: widest split target (2k = 64), and a padded one (2k = 10 -> 16)
    "bf16_d1536_k32_fused": gen.custom_config("t11", blocks=1, d=1536, n=2000, micro=1000, C=5, k=32, r_a=8),
    "bf16_d1280_k5_fused": gen.custom_config("t12", blocks=2, d=1280, n=1600, micro=800, C=3, k=5, r_a=2),
    # 2k = 128 > 64: the cross statistic as cross tiles of the direct-load Gram launch (half of
    # each cross tile's columns past the split targets)
    "bf16_d1024_k64": gen.custom_config("t13", blocks=1, d=1024, n=1200, C=3, k=64, r_a=8),
    # 2k = 256: cross tiles at their full width, ragged d against 256-wide tiles, two blocks,
    # two micro-batches; 128 right-hand sides in the solve and the large truncation core
    "bf16_d1288_k128": gen.custom_config("t16", blocks=2, d=1288, n=2700, micro=1500, C=6, k=128, r_a=16),
    # 19 x 19 tile rows plus 19 cross tiles per block (at least 24 tiles per XCD): the Gram launch
    # in its block-synchronous order over all eight XCDs, two micro-batches
    "bf16_d4864_k64_sync": gen.custom_config("t18", blocks=1, d=4864, n=5200, micro=2600, C=5, k=64, r_a=8),
    # 13 x 13 tile rows plus 13 cross tiles per block and two blocks: XCD groups of four, one
    # block per group
    "bf16_d3328_k64_groups": gen.custom_config("t19", blocks=2, d=3328, n=3500, C=4, k=64, r_a=8),
    # fp32 mode with fewer tokens than features (null space amplified by 1/lambda)
    "fp32_n150_d200": gen.custom_config("t3", blocks=2, d=200, n=150, C=2, k=8, r_a=8, mode="fp32",
                                        x_dist="gauss_outlier", n_outlier=3, outlier_scale=20.0, logit_std=2.0),
    # large label set (online-softmax kernel), bf16 logits and credit factor, real truncation 64 -> 32
    "vocab3000": gen.custom_config("t4", blocks=1, d=256, n=600, C=3000, k=64, r_a=32, logit_std=2.0,
                                   logit_dtype="bf16", a_dtype="bf16"),
    # k > 64 on a small label set goes through the large-vocabulary kernel too
    "k96": gen.custom_config("t5", blocks=1, d=320, n=400, C=7, k=96, r_a=16),
}


@pytest.mark.parametrize("name", list(CASES))
def test_block_step_parity(name):
    cfg = CASES[name]
    log(f"case {name}: d={cfg.d} n={cfg.n} C={cfg.C} k={cfg.k} blocks={cfg.blocks} mode={cfg.mode}")
    xs, zs, ys, As, Bs = host_inputs(cfg, range(cfg.blocks))
    g = run_gpu(cfg, xs, zs, ys, As, Bs)
    assert np.all(g["info"] == 0) and np.all(g["info_err"] == 0)
    for b in range(cfg.blocks):
        o = run_oracle(cfg, xs[b], zs, ys, As[b], Bs[b])
        _compare(cfg, g, o, b, f"{name}[block {b}]")


def test_k96_credit_coordinates():
    """k = 96: head error (the streaming kernel: k > 64 with an fp32 A~) and ||Q||^2."""
    import torch
    from paper_2608_03020_amd import loca
    import oracle
    cfg = CASES["k96"]
    xs, zs, ys, As, Bs = host_inputs(cfg, [0])
    log("case k96 statistics")
    from paper_2608_03020_amd.step import BlockStep
    st = BlockStep(cfg, 1)
    x = padded_rows(np.stack([np.concatenate(xs[0])]))
    st.reset()
    st.micro_batch(x, to_dev(zs[0]), to_dev(ys[0]), to_dev(np.stack(As)), to_dev(np.stack(Bs)))
    torch.cuda.synchronize()
    E = oracle.head_error(zs[0], ys[0])
    Y, Q = oracle.credit(E, As[0], Bs[0])
    assert rel(st.Y[0].cpu().numpy(), Y) < 1e-5
    mbv = loca.mb_view(st.mb)
    assert abs(mbv["sum_q2"][0] - np.sum(Q ** 2)) / np.sum(Q ** 2) < 1e-5


@pytest.mark.parametrize("k,blocks", [(24, 1), (64, 1), (32, 2)])
def test_large_vocab_padded_logit_rows(k, blocks):
    """A large vocabulary through the matrix-core product with bf16 logits in a padded buffer
    (3001 classes in rows 3008 wide): the softmax statistics' 8-wide chunks and their
    one-logit tail, Y = E A~ and ||Q||^2 from the credit Gram padded to 32 (k = 24: padding
    inside the register rows) or 64; two blocks of k = 32 share one 64-column product tile."""
    import torch
    from paper_2608_03020_amd import loca
    from paper_2608_03020_amd.step import BlockStep
    import oracle
    cfg = gen.custom_config("t17", blocks=blocks, d=256, n=300, C=3001, k=k, r_a=8, logit_std=2.0,
                            logit_dtype="bf16", a_dtype="bf16")
    xs, zs, ys, As, Bs = host_inputs(cfg, list(range(blocks)))
    log(f"case vocab 3001 in rows of 3008, k = {k}, {blocks} block(s)")
    st = BlockStep(cfg, blocks)
    st.reset()
    z = zs[0]
    n = z.shape[0]
    buf = np.zeros((n, 3008), np.uint16)
    buf[:, :3001] = z
    zd = to_dev(buf)[:, :3001]
    assert zd.stride(0) == 3008
    loca.loca_error_targets(zd, to_dev(ys[0]), to_dev(np.stack(As)), to_dev(np.stack(Bs)), st.Y[:, :n], st.mb,
                            st.info_err[:1], st.ws)
    torch.cuda.synchronize()
    assert int(st.info_err[0].item()) == 0
    E = oracle.head_error(gen.as_f64(z, "bf16"), ys[0])
    q2 = loca.mb_view(st.mb)["sum_q2"]
    for b in range(blocks):
        Y, Q = oracle.credit(E, gen.as_f64(As[b], "bf16"), np.asarray(Bs[b], np.float64))
        ey = rel(st.Y[b, :n].cpu().numpy(), Y)
        eq = abs(q2[b] - np.sum(Q ** 2)) / np.sum(Q ** 2)
        log(f"block {b}: Y rel err {ey:.2e}, ||Q||^2 rel err {eq:.2e}")
        assert ey < 1e-4 and eq < 2e-4


@pytest.mark.parametrize("C,k,ldz,dt", [(9, 24, 9, "f32"), (17, 64, 24, "bf16"), (64, 32, 64, "f32"), (5, 64, 8, "bf16")])
def test_register_head_many_classes(C, k, ldz, dt):
    """The register head (C <= 64 classes, k <= 64) with its logits in chunks of 8 classes:
    one chunk plus a tail of 1 (C = 9), three chunks in a padded buffer (C = 17 in rows of
    24), eight chunks (C = 64), and C = 5 in rows of 8; 300 tokens (a ragged workgroup), two
    blocks; E, Y and ||Q||^2 against the oracle."""
    import torch
    from paper_2608_03020_amd import loca
    from paper_2608_03020_amd.step import BlockStep
    import oracle
    cfg = gen.custom_config(f"head{C}", blocks=2, d=256, n=300, C=C, k=k, r_a=8, logit_std=2.0,
                            logit_dtype=dt, a_dtype="f32")
    xs, zs, ys, As, Bs = host_inputs(cfg, [0, 1])
    log(f"case register head: C={C} k={k} logits {dt} in rows of {ldz}, 2 blocks")
    st = BlockStep(cfg, 2)
    st.reset()
    z = zs[0]
    n = z.shape[0]
    buf = np.zeros((n, ldz), z.dtype)
    buf[:, :C] = z
    zd = to_dev(buf)[:, :C]
    e_out = torch.full((n, C), float("nan"), device="cuda")
    loca.loca_error_targets(zd, to_dev(ys[0]), to_dev(np.stack(As)), to_dev(np.stack(Bs)), st.Y[:, :n], st.mb,
                            st.info_err[:1], st.ws, e_out=e_out)
    torch.cuda.synchronize()
    assert int(st.info_err[0].item()) == 0
    E = oracle.head_error(gen.as_f64(z, dt), ys[0])
    ee = rel(e_out.cpu().numpy(), E)
    q2 = loca.mb_view(st.mb)["sum_q2"]
    for b in range(2):
        Y, Q = oracle.credit(E, np.asarray(As[b], np.float64), np.asarray(Bs[b], np.float64))
        ey = rel(st.Y[b, :n].cpu().numpy(), Y)
        eq = abs(q2[b] - np.sum(Q ** 2)) / np.sum(Q ** 2)
        log(f"block {b}: E rel err {ee:.2e}, Y rel err {ey:.2e}, ||Q||^2 rel err {eq:.2e}")
        assert ee < 1e-5 and ey < 1e-5 and eq < 1e-5


def test_dense_targets_and_cross_statistic():
    """T = -eta_bar Y B~ (dense) and Z = X^T T = K B~ against the oracle's dense Z."""
    import torch
    from paper_2608_03020_amd import loca
    cfg = CASES["bf16_d600"]
    xs, zs, ys, As, Bs = host_inputs(cfg, [0])
    g = run_gpu(cfg, xs, zs, ys, As, Bs, want_dense=False)
    o = run_oracle(cfg, xs[0], zs, ys, As[0], Bs[0])
    Z_gpu = g["K"][0].astype(np.float64) @ np.asarray(Bs[0], np.float64)
    log("dense Z rel err", rel(Z_gpu, o["Z"]))
    assert rel(Z_gpu, o["Z"]) <= TOL["bf16"]
    # dense T of the last micro-batch
    m = cfg.n_micro - 1
    y = torch.from_numpy(g["Y"][m]).cuda()
    mbt = torch.from_numpy(np.stack([[g["mb"][m]["sum_q2"][0], g["mb"][m]["sum_x2"][0], g["mb"][m]["eta_bar"][0],
                                      np.int64(g["mb"][m]["n"][0]).view(np.float64)]])).cuda()
    T = torch.empty((1, y.shape[1], cfg.d), dtype=torch.float32, device="cuda")
    loca.loca_dense_targets(y, mbt, torch.from_numpy(np.stack(Bs)).cuda(), T)
    torch.cuda.synchronize()
    assert rel(T[0].cpu().numpy(), o["T"][m]) <= 1e-5


def test_ridge_solve_from_oracle_statistics():
    """The solve alone, fed the oracle's statistics: M = (S + lam I)^{-1} K per lambda, and dense W."""
    import torch
    from paper_2608_03020_amd import loca
    cfg = gen.custom_config("t6", blocks=1, d=777, n=2000, C=5, k=32, r_a=8, lambdas=(1e-3, 1e-2, 1e-1))
    xs, zs, ys, As, Bs = host_inputs(cfg, [0])
    o = run_oracle(cfg, xs[0], zs, ys, As[0], Bs[0])
    S = torch.from_numpy(o["S"].astype(np.float32))[None].cuda()
    K = torch.from_numpy(o["K"].astype(np.float32))[None].cuda()
    M = torch.empty((1, 3, cfg.d, cfg.k), dtype=torch.float32, device="cuda")
    W = torch.empty((1, 3, cfg.d, cfg.d), dtype=torch.float32, device="cuda")
    info = torch.zeros(3, dtype=torch.int32, device="cuda")
    ws = loca.alloc_workspace(loca.workspace_size(loca.LOCA_OP_RIDGE_SOLVE, 1, 0, cfg.d, cfg.k, n_lambda=3))
    B = torch.from_numpy(Bs[0])[None].cuda()
    loca.loca_ridge_solve(S, K, cfg.lambdas, M, info, ws, credit_b=B, w_dense_out=W)
    torch.cuda.synchronize()
    assert np.all(info.cpu().numpy() == 0)
    for l, sol in enumerate(o["solves"]):
        em, ew = rel(M[0, l].cpu().numpy(), sol["M"]), rel(W[0, l].cpu().numpy(), sol["W"])
        log(f"solve lam={cfg.lambdas[l]}: M {em:.2e} W {ew:.2e}")
        assert em < 2e-4 and ew < 2e-4


def test_ridge_solve_fp64_and_nonpd_pivot():
    """fp64 solve of an exactly known system, and the potrf-style pivot report."""
    import torch
    from paper_2608_03020_amd import loca
    rng = np.random.default_rng(0)
    d, k = 130, 5
    Xr = rng.normal(size=(300, d))
    S = Xr.T @ Xr
    K = rng.normal(size=(d, k))
    lam = 0.5
    Mref = np.linalg.solve(S + lam * np.eye(d), K)
    St = torch.from_numpy(S)[None].cuda()
    Kt = torch.from_numpy(K)[None].cuda()
    M = torch.empty((1, 1, d, k), dtype=torch.float32, device="cuda")
    info = torch.zeros(1, dtype=torch.int32, device="cuda")
    ws = loca.alloc_workspace(loca.workspace_size(loca.LOCA_OP_RIDGE_SOLVE, 1, 0, d, k, n_lambda=1,
                                                  acc=loca.LOCA_F64))
    loca.loca_ridge_solve(St, Kt, [lam], M, info, ws)
    torch.cuda.synchronize()
    assert info.item() == 0
    assert rel(M[0, 0].cpu().numpy(), Mref) < 1e-6  # fp32 output rounding
    # a negative diagonal entry at index 70 is the first non-positive pivot (1-based 71)
    S2 = S.copy()
    S2[70, 70] = -1e6
    loca.loca_ridge_solve(torch.from_numpy(S2)[None].cuda(), Kt, [lam], M, info, ws)
    torch.cuda.synchronize()
    assert info.item() == 71


@pytest.mark.parametrize("kp,r", [(40, 12), (64, 30), (96, 40)])
def test_truncation_rank_deficient_right_factor(kp, r):
    """R with repeated rows (R R^T singular): the core (for kp <= 64, and the one for
    64 < kp <= 128) takes the eigendecomposition of R R^T instead of its Cholesky factor;
    W_r against the oracle's dense SVD."""
    import torch
    import oracle
    from paper_2608_03020_amd import loca
    d = 180
    rng = np.random.default_rng(2)
    log(f"case truncation_rank_deficient: d={d} kp={kp} r_a={r}")
    Mh = rng.normal(size=(d, kp)).astype(np.float32)
    half = rng.normal(size=(kp // 2, d)).astype(np.float32)
    Rh = np.concatenate([half, half])
    Wr_o, s_o = oracle.truncate_dense(Mh.astype(np.float64) @ Rh.astype(np.float64), r)
    a = torch.empty((1, r, d), device="cuda")
    b = torch.empty((1, d, r), device="cuda")
    s = torch.empty((1, kp), device="cuda")
    W = torch.empty((1, d, d), device="cuda")
    info = torch.zeros(1, dtype=torch.int32, device="cuda")
    ws = loca.alloc_workspace(loca.workspace_size(loca.LOCA_OP_LOWRANK_TRUNCATE, 1, 0, d, kp, r_a=r))
    loca.loca_lowrank_truncate(torch.from_numpy(Mh)[None].cuda(), torch.from_numpy(Rh)[None].cuda(), r, a, b, s,
                               info, ws, w_dense_out=W)
    torch.cuda.synchronize()
    e_w = rel(W[0].cpu().numpy(), Wr_o)
    e_s = rel(s[0].cpu().numpy()[:kp // 2], s_o[:kp // 2])
    log(f"truncation (rank-deficient R): W_r {e_w:.2e} sigma {e_s:.2e}")
    assert e_w < 1e-5 and e_s < 1e-5


@pytest.mark.parametrize("d,kp,r", [(200, 24, 10), (200, 64, 32), (130, 63, 20), (96, 2, 1), (200, 96, 40),
                                    (230, 127, 64), (150, 128, 16)])
def test_truncation_matches_explicit_svd(d, kp, r):
    """Eckart-Young truncation of W = M B~ against the oracle's dense SVD (d <= 256): the
    fp64-LDS core for kp <= 64 (its largest kp, an odd kp padded, kp = 2) and the core with
    float eigenvectors for kp > 64 (odd kp padded, the largest kp and rank)."""
    import torch
    import oracle
    from paper_2608_03020_amd import loca
    rng = np.random.default_rng(1)
    log(f"case truncation: d={d} kp={kp} r_a={r}")
    Mh = rng.normal(size=(d, kp)).astype(np.float32)
    Rh = rng.normal(size=(kp, d)).astype(np.float32)
    Wr_o, s_o = oracle.truncate_dense(Mh.astype(np.float64) @ Rh.astype(np.float64), r)
    Mt = torch.from_numpy(Mh)[None].cuda()
    Rt = torch.from_numpy(Rh)[None].cuda()
    a = torch.empty((1, r, d), device="cuda")
    b = torch.empty((1, d, r), device="cuda")
    s = torch.empty((1, kp), device="cuda")
    W = torch.empty((1, d, d), device="cuda")
    info = torch.zeros(1, dtype=torch.int32, device="cuda")
    ws = loca.alloc_workspace(loca.workspace_size(loca.LOCA_OP_LOWRANK_TRUNCATE, 1, 0, d, kp, r_a=r))
    loca.loca_lowrank_truncate(Mt, Rt, r, a, b, s, info, ws, w_dense_out=W)
    torch.cuda.synchronize()
    e_w = rel(W[0].cpu().numpy(), Wr_o)
    e_s = rel(s[0].cpu().numpy(), s_o[:kp])
    A = a[0].cpu().numpy().astype(np.float64)
    log(f"truncation: W_r {e_w:.2e} sigma {e_s:.2e} orth {np.abs(A @ A.T - np.eye(r)).max():.2e}")
    assert e_w < 1e-5 and e_s < 1e-5
    assert np.abs(A @ A.T - np.eye(r)).max() < 1e-5
    np.testing.assert_allclose(A.T @ b[0].cpu().numpy().T, W[0].cpu().numpy(), atol=1e-4 * np.abs(Wr_o).max())


@pytest.mark.parametrize("kp,r,rank", [(64, 32, 5), (96, 40, 5), (64, 32, 0), (32, 16, 15)])
def test_truncation_low_rank_product(kp, r, rank):
    """W = M B~ of rank below r_a (a label set of six classes makes Y, hence K and M, of rank
    5; M = 0 gives W = 0): the directions with weight from the tridiagonal path, the others
    numerically zero, so their b_out columns are zero and their a_out rows an orthonormal
    completion; W_r and the leading sigma against the oracle's dense SVD."""
    import torch
    import oracle
    from paper_2608_03020_amd import loca
    d = 300
    rng = np.random.default_rng(5 + rank)
    log(f"case truncation_low_rank: d={d} kp={kp} r_a={r} rank={rank}")
    Mh = (rng.normal(size=(d, rank)) @ rng.normal(size=(rank, kp))).astype(np.float32)
    Rh = rng.normal(size=(kp, d)).astype(np.float32)
    Wr_o, s_o = oracle.truncate_dense(Mh.astype(np.float64) @ Rh.astype(np.float64), r)
    a = torch.empty((1, r, d), device="cuda")
    b = torch.empty((1, d, r), device="cuda")
    s = torch.empty((1, kp), device="cuda")
    W = torch.empty((1, d, d), device="cuda")
    info = torch.zeros(1, dtype=torch.int32, device="cuda")
    ws = loca.alloc_workspace(loca.workspace_size(loca.LOCA_OP_LOWRANK_TRUNCATE, 1, 0, d, kp, r_a=r))
    loca.loca_lowrank_truncate(torch.from_numpy(Mh)[None].cuda(), torch.from_numpy(Rh)[None].cuda(), r, a, b, s,
                               info, ws, w_dense_out=W)
    torch.cuda.synchronize()
    A = a[0].cpu().numpy().astype(np.float64)
    B = b[0].cpu().numpy()
    orth = np.abs(A @ A.T - np.eye(r)).max()
    if rank == 0:
        log(f"truncation (W = 0): |W_r| {np.abs(W[0].cpu().numpy()).max():.1e} |sigma| "
            f"{np.abs(s[0].cpu().numpy()).max():.1e} |b_out| {np.abs(B).max():.1e} orth {orth:.2e}")
        assert np.abs(W[0].cpu().numpy()).max() == 0.0 and np.abs(s[0].cpu().numpy()).max() == 0.0
        assert np.abs(B).max() == 0.0 and orth < 1e-6
        return
    e_w = rel(W[0].cpu().numpy(), Wr_o)
    e_s = rel(s[0].cpu().numpy()[:rank], s_o[:rank])
    log(f"truncation (rank {rank}): W_r {e_w:.2e} sigma {e_s:.2e} orth {orth:.2e} "
        f"dead b_out {np.abs(B[:, rank:]).max():.1e}")
    assert e_w < 1e-5 and e_s < 1e-5
    assert orth < 1e-5
    assert np.abs(B[:, rank:]).max() <= 1e-6 * np.abs(B[:, :rank]).max()


@pytest.mark.parametrize("kp,r", [(64, 32), (32, 8), (96, 32)])
def test_truncation_repeated_leading_values(kp, r):
    """Repeated singular values among the r kept (a triple and a pair): the eigenvectors of the
    repeated eigenvalues cannot be told apart by the tridiagonal solves, so the core's check
    sends the eigensolve to Jacobi (both cores).  M and B~ from Hadamard matrices / 8
    (orthogonal and exact in float; two blocks on disjoint rows past 64 columns), so that
    W = M B~ has exactly the chosen singular values; W_r against the oracle's dense SVD (the
    kept subspace is unique: sigma_r > sigma_{r+1})."""
    import torch
    import oracle
    from scipy.linalg import hadamard
    from paper_2608_03020_amd import loca
    d = 150
    log(f"case truncation_repeated: d={d} kp={kp} r_a={r}")
    H = hadamard(64).astype(np.float64) / 8.0  # orthogonal, exact in float
    Q = np.zeros((128, kp))  # orthonormal columns: H's, then H's again on rows 64..127
    Q[:64, :min(kp, 64)] = H[:, :min(kp, 64)]
    if kp > 64:
        Q[64:, 64:] = H[:, :kp - 64]
    sig = np.concatenate([[6.0, 6.0, 6.0, 5.0, 5.0], np.linspace(4.0, 0.5, kp - 5)])
    Mh = np.zeros((d, kp), dtype=np.float32)
    Mh[:128] = (Q * sig).astype(np.float32)
    Rh = np.zeros((kp, d), dtype=np.float32)
    Rh[:, 10:10 + 128] = Q.T.astype(np.float32)
    Wd = Mh.astype(np.float64) @ Rh.astype(np.float64)
    Wr_o, s_o = oracle.truncate_dense(Wd, r)
    assert np.allclose(s_o[:kp], sig, rtol=1e-6) and np.ptp(s_o[:3]) < 1e-12 * s_o[0]
    a = torch.empty((1, r, d), device="cuda")
    b = torch.empty((1, d, r), device="cuda")
    s = torch.empty((1, kp), device="cuda")
    W = torch.empty((1, d, d), device="cuda")
    info = torch.zeros(1, dtype=torch.int32, device="cuda")
    ws = loca.alloc_workspace(loca.workspace_size(loca.LOCA_OP_LOWRANK_TRUNCATE, 1, 0, d, kp, r_a=r))
    loca.loca_lowrank_truncate(torch.from_numpy(Mh)[None].cuda(), torch.from_numpy(Rh)[None].cuda(), r, a, b, s,
                               info, ws, w_dense_out=W)
    torch.cuda.synchronize()
    e_w = rel(W[0].cpu().numpy(), Wr_o)
    e_s = rel(s[0].cpu().numpy(), s_o[:kp])
    A = a[0].cpu().numpy().astype(np.float64)
    log(f"truncation (repeated leading values): W_r {e_w:.2e} sigma {e_s:.2e} "
        f"orth {np.abs(A @ A.T - np.eye(r)).max():.2e}")
    assert e_w < 1e-5 and e_s < 1e-5
    assert np.abs(A @ A.T - np.eye(r)).max() < 1e-5


@pytest.mark.parametrize("d,n,k,r_a,mode", [(300, 500, 16, 8, "bf16"), (1100, 2400, 48, 40, "bf16"),
                                             (130, 700, 64, 64, "bf16"), (200, 150, 16, 16, "fp32")])
def test_projected_form_matches_oracle(d, n, k, r_a, mode):
    """Paper-literal projected solve (random A_l): B* = C_l (G_l + lam I)^{-1}; panels of the
    symmetric S with ragged edges, r_a on both sides of 32, fp32 and fp64 statistics."""
    cfg = gen.custom_config("t7", blocks=2, d=d, n=n, C=4, k=k, r_a=r_a, lambdas=(1e-2, 1.0), mode=mode,
                            x_dist="gauss_outlier" if mode == "fp32" else "rms_outlier")
    log(f"case projected d={d} n={n} k={k} r_a={r_a} {mode}")
    xs, zs, ys, As, Bs = host_inputs(cfg, range(2))
    proj = [gen.gen_adapter_projection(cfg, b) for b in range(2)]
    g = run_gpu(cfg, xs, zs, ys, As, Bs, want_dense=False, proj=proj)
    for b in range(2):
        o = run_oracle(cfg, xs[b], zs, ys, As[b], Bs[b], proj=proj[b])
        for l, sol in enumerate(o["solves"]):
            e = rel(g["B_proj"][b, l], sol["B_proj"])
            log(f"projected block {b} lam {cfg.lambdas[l]}: {e:.2e}")
            assert e <= TOL[mode]


def test_degenerate_single_class_and_zero_eta():
    """C = 1 gives E = 0, so Q = 0, eta_bar = 0 and the adapter is zero (frozen model)."""
    cfg = gen.custom_config("t8", blocks=1, d=40, n=33, C=1, k=4, r_a=2)
    xs, zs, ys, As, Bs = host_inputs(cfg, [0])
    g = run_gpu(cfg, xs, zs, ys, As, Bs)
    assert np.all(g["mb"][0]["eta_bar"] == 0.0)
    assert np.all(g["K"] == 0.0) and np.all(g["M"] == 0.0) and np.all(g["W_r"] == 0.0)
    o = run_oracle(cfg, xs[0], zs, ys, As[0], Bs[0])
    assert rel(g["S"][0][np.triu_indices(40)], o["S"][np.triu_indices(40)]) < 1e-6


def test_tiny_width_and_single_token():
    """d = 1 (one feature, ldx padded to 8) and a single-token micro-batch."""
    import torch
    from paper_2608_03020_amd import loca
    import oracle
    rng = np.random.default_rng(2)
    for n, d in [(1, 1), (1, 9), (37, 1)]:
        log(f"case tiny n={n} d={d}")
        ld = 8 * ((d + 7) // 8)
        xh = gen.bf16_bits(rng.normal(size=(n, d)).astype(np.float32))
        xpad = np.zeros((1, n, ld), np.uint16)
        xpad[0, :, :d] = xh
        x = to_dev(xpad)[:, :, :d]
        k = 1
        y = torch.from_numpy(rng.normal(size=(1, n, k)).astype(np.float32)).cuda()
        mb = loca.new_mb(1)
        mb[0, 0] = 1.0  # sum_q2 = 1
        S = torch.zeros((1, d, d), device="cuda")
        K = torch.zeros((1, d, k), device="cuda")
        ws = loca.alloc_workspace(loca.workspace_size(loca.LOCA_OP_ACCUMULATE_STATS, 1, n, d, k))
        loca.loca_accumulate_stats(x, y, 0.5, mb, S, K, ws)
        torch.cuda.synchronize()
        xf = gen.as_f64(xh, "bf16")
        So = oracle.gram_acc(xf)
        sx = float(np.sum(xf ** 2))
        eb = 0.5 * np.sqrt(sx / 1.0)
        Ko = oracle.cross_acc(xf, -eb * y[0].cpu().numpy().astype(np.float64))
        iu = np.triu_indices(d)
        assert rel(S[0].cpu().numpy()[iu], So[iu]) < 1e-6
        assert rel(K[0].cpu().numpy(), Ko) < 1e-5
        assert abs(loca.mb_view(mb)["eta_bar"][0] - eb) < 1e-6 * eb


@pytest.mark.parametrize("d,k,mode,weighted", [(1040, 8, "bf16", False), (1040, 40, "bf16", True),
                                               (1024, 64, "bf16", False), (200, 24, "bf16", True),
                                               (100, 12, "fp32", True)])
def test_stats_overwrite_equals_cleared_accumulation(d, k, mode, weighted):
    """The overwrite flag (the first micro-batch of a step) leaves S's upper triangle, K and
    the micro-batch records bit for bit as the accumulating call on zeroed S and K, without
    reading the old contents (NaN here); a second, accumulating micro-batch keeps them
    equal.  Paths: the direct-to-LDS Gram kernel with the cross statistic fused (k = 8)
    and as cross tiles (k = 40, 64), the register-staged kernel (d = 200), the fp64 kernel."""
    import torch
    from paper_2608_03020_amd import loca
    nb, n = 2, 300
    log(f"case stats overwrite: d={d} k={k} mode={mode} weighted={weighted}")
    g = torch.Generator(device="cuda")
    g.manual_seed(d + k)
    xt, acc_t = (torch.bfloat16, torch.float32) if mode == "bf16" else (torch.float32, torch.float64)
    acc = loca.LOCA_F32 if mode == "bf16" else loca.LOCA_F64
    ld = (d + 7) // 8 * 8
    xs = [torch.randn((nb, n, ld), generator=g, device="cuda").to(xt)[:, :, :d] for _ in range(2)]
    ys = [torch.randn((nb, n, k), generator=g, device="cuda") for _ in range(2)]
    aws = [torch.rand(n, generator=g, device="cuda") if weighted else None for _ in range(2)]
    ws = loca.alloc_workspace(loca.workspace_size(loca.LOCA_OP_ACCUMULATE_STATS, nb, n, d, k, acc=acc))
    out = []
    for ovw in (False, True):
        fill = float("nan") if ovw else 0.0
        S = torch.full((nb, d, d), fill, dtype=acc_t, device="cuda")
        K = torch.full((nb, d, k), fill, dtype=acc_t, device="cuda")
        res = []
        for m in range(2):
            mb = loca.new_mb(nb)
            mb[:, 0] = 1.0 + m  # sum_q2
            loca.loca_accumulate_stats(xs[m], ys[m], 0.5, mb, S, K, ws, a_w=aws[m], overwrite=ovw and m == 0)
            torch.cuda.synchronize()
            res.append((torch.triu(S).cpu().numpy(), K.cpu().numpy(), mb.cpu().numpy()))
        out.append(res)
    for m in range(2):
        for a, b in zip(out[0][m], out[1][m]):
            assert np.array_equal(a, b), m
    assert not np.isnan(out[1][1][0]).any() and not np.isnan(out[1][1][1]).any()


@pytest.mark.parametrize("C,k,ldt,adt", [(5, 32, "f32", "f32"), (4, 5, "f32", "f32"), (3001, 24, "f32", "f32"),
                                         (3001, 32, "bf16", "bf16"), (3001, 96, "bf16", "bf16"), (70, 72, "f32", "bf16")])
def test_precomputed_credit_gram_gives_the_same_bits(C, k, ldt, adt):
    """loca_error_targets with B~ B~^T from loca_credit_gram equals the call that forms it,
    bit for bit, on every path (small label sets, the streaming kernel, the vocabulary
    product with k <= 64 and k > 64) and padded Gram widths (k = 5, 24, 72)."""
    import torch
    from paper_2608_03020_amd import loca
    n, d, nb = 700, 200, 3
    g = torch.Generator(device="cuda")
    g.manual_seed(C + k)
    zt = torch.bfloat16 if ldt == "bf16" else torch.float32
    ld = (C + 7) // 8 * 8
    zbuf = torch.zeros((n, ld), device="cuda", dtype=zt)
    zbuf[:, :C] = (torch.randn((n, C), generator=g, device="cuda") * 2).to(zt)
    z = zbuf[:, :C]
    y = torch.randint(0, C, (n,), generator=g, device="cuda", dtype=torch.int32)
    A = (torch.randn((nb, C, k), generator=g, device="cuda") / np.sqrt(k)).to(
        torch.bfloat16 if adt == "bf16" else torch.float32)
    B = torch.randn((nb, k, d), generator=g, device="cuda") / np.sqrt(k)
    aw = torch.rand(n, generator=g, device="cuda")
    ws = loca.alloc_workspace(max(loca.workspace_size(loca.LOCA_OP_ERROR_TARGETS, nb, n, d, k, C),
                                  loca.workspace_size(loca.LOCA_OP_CREDIT_GRAM, nb, 0, d, k)))
    G = loca.new_credit_gram(nb, k)
    G.fill_(float("nan"))
    loca.loca_credit_gram(B, G, ws)
    out = []
    for gram in (None, G):
        Y = torch.full((nb, n, k), float("nan"), device="cuda")
        mb = loca.new_mb(nb)
        info = torch.full((1,), 5, dtype=torch.int32, device="cuda")
        loca.loca_error_targets(z, y, A, B, Y, mb, info, ws, a_w=aw, credit_gram=gram)
        torch.cuda.synchronize()
        assert info.item() == 0
        out.append((Y.cpu().numpy(), mb.cpu().numpy()))
    assert not np.isnan(out[1][0]).any()
    assert np.array_equal(out[0][0], out[1][0]) and np.array_equal(out[0][1], out[1][1])
    Gh = G.cpu().numpy()
    ldg = Gh.shape[-1]
    Bh = B.double().cpu().numpy()
    for b in range(nb):
        ref = Bh[b] @ Bh[b].T
        assert np.abs(Gh[b, :k, :k] - ref).max() <= 1e-12 * np.abs(ref).max()
        assert np.all(Gh[b, k:, :] == 0) and np.all(Gh[b, :, k:] == 0) and ldg >= k


def test_out_of_range_label_reported():
    import torch
    from paper_2608_03020_amd import loca
    n, C, k, d = 300, 4, 8, 16
    z = torch.randn((n, C), device="cuda")
    y = torch.randint(0, C, (n,), dtype=torch.int32, device="cuda")
    y[123] = 9
    y[200] = -1
    A = torch.randn((1, C, k), device="cuda")
    B = torch.randn((1, k, d), device="cuda")
    Y = torch.empty((1, n, k), device="cuda")
    mb = loca.new_mb(1)
    info = torch.zeros(1, dtype=torch.int32, device="cuda")
    ws = loca.alloc_workspace(loca.workspace_size(loca.LOCA_OP_ERROR_TARGETS, 1, n, d, k, C))
    loca.loca_error_targets(z, y, A, B, Y, mb, info, ws)
    torch.cuda.synchronize()
    assert info.item() == 124


def test_statistics_deterministic_and_resumable():
    """Same inputs in the same order give bitwise-equal S and K; stopping after two
    micro-batches, saving S, K to the host and resuming gives the same bits."""
    import torch
    cfg = gen.custom_config("t9", blocks=2, d=520, n=1600, micro=400, C=5, k=16, r_a=4)
    xs, zs, ys, As, Bs = host_inputs(cfg, range(2))
    from paper_2608_03020_amd.step import BlockStep
    x_all = padded_rows(np.stack([np.concatenate(xb) for xb in xs]))
    z_all, y_all = to_dev(np.concatenate(zs)), to_dev(np.concatenate(ys))
    A, B = to_dev(np.stack(As)), to_dev(np.stack(Bs))

    def run(split=None):
        st = BlockStep(cfg, 2)
        st.reset()
        for m in range(cfg.n_micro):
            if split is not None and m == split:
                S_h, K_h = st.S.cpu().numpy().copy(), st.K.cpu().numpy().copy()
                st = BlockStep(cfg, 2)
                st.resume(torch.from_numpy(S_h), torch.from_numpy(K_h), m)
            lo, hi = cfg.micro_rows(m)
            st.micro_batch(x_all[:, lo:hi], z_all[lo:hi], y_all[lo:hi], A, B)
        torch.cuda.synchronize()
        return st.S.cpu().numpy(), st.K.cpu().numpy()

    S1, K1 = run()
    S2, K2 = run()
    S3, K3 = run(split=2)
    iu = np.triu_indices(cfg.d)
    assert np.array_equal(S1[:, iu[0], iu[1]], S2[:, iu[0], iu[1]]) and np.array_equal(K1, K2)
    assert np.array_equal(S1[:, iu[0], iu[1]], S3[:, iu[0], iu[1]]) and np.array_equal(K1, K3)


@pytest.mark.parametrize("mode", ["bf16", "fp32", "bf16_kp88"])
def test_outer_step_with_current_adapter(mode):
    """Theorem S6.1 past the first outer step: (S + lam I) W = S W_prev + Z with a current
    adapter W_prev = Lp Rp != 0, solved in factored form M = (S + lam I)^{-1} [S Lp | K],
    W = M [Rp; B~], and truncated to rank r_a from its factors (kp = r_prev + k)."""
    import torch
    import oracle
    from paper_2608_03020_amd.step import BlockStep
    if mode == "bf16":
        cfg = gen.custom_config("t14", blocks=2, d=288, n=900, micro=500, C=4, k=16, r_a=8, lambdas=(1e-2, 0.1))
        r_prev, tol = 6, 2e-3
    elif mode == "bf16_kp88":  # r_prev + k = 88 > 64: the packed-LDS truncation
        cfg = gen.custom_config("t14b", blocks=2, d=300, n=1200, micro=700, C=6, k=48, r_a=24, lambdas=(1e-2,))
        r_prev, tol = 40, 2e-3
    else:
        cfg = gen.custom_config("t14f", blocks=2, d=150, n=300, micro=180, C=3, k=8, r_a=6, lambdas=(1e-2, 0.1),
                                mode="fp32", x_dist="gauss_outlier")
        r_prev, tol = 5, 1e-5
    blocks = [0, 1]
    log(f"case outer_step {mode}: d={cfg.d} n={cfg.n} k={cfg.k} r_prev={r_prev} r_a={cfg.r_a} lambdas={cfg.lambdas}")
    xs, zs, ys, As, Bs = host_inputs(cfg, blocks)
    xf = [[gen.as_f64(x, "f32" if mode == "fp32" else "bf16") for x in xs[b]] for b in blocks]
    zf = [gen.as_f64(z, cfg.logit_dtype) for z in zs]
    frozen = [oracle.block_step(xf[b], zf, ys, gen.as_f64(As[b], cfg.a_dtype), np.asarray(Bs[b], np.float64),
                                cfg.eta, (cfg.lambdas[0],), cfg.r_a) for b in blocks]
    Lps, Rps = [], []
    for b in blocks:  # current adapter scaled so that S W_prev and Z are of one size
        lp, rp = gen.gen_current_adapter(cfg, b, r_prev)
        Wp = lp.astype(np.float64) @ rp.astype(np.float64)
        scale = np.linalg.norm(frozen[b]["Z"]) / np.linalg.norm(frozen[b]["S"] @ Wp)
        Lps.append(lp)
        Rps.append((rp * np.float32(scale)).astype(np.float32))
    dev = "cuda"
    step = BlockStep(cfg, len(blocks), dev, r_prev=r_prev)
    x_all = padded_rows(np.stack([np.concatenate(xb, axis=0) for xb in xs]), dev)
    z_all, y_all = to_dev(np.concatenate(zs, axis=0), dev), to_dev(np.concatenate(ys, axis=0), dev)
    A, B = to_dev(np.stack(As), dev), to_dev(np.stack(Bs), dev)
    step.reset()
    for m in range(cfg.n_micro):
        lo, hi = cfg.micro_rows(m)
        step.micro_batch(x_all[:, lo:hi], z_all[lo:hi], y_all[lo:hi], A, B, keep_log=True)
    lp_d, rp_d = to_dev(np.stack(Lps), dev), to_dev(np.stack(Rps), dev)
    step.solve(B, lp=lp_d, rp=rp_d)
    torch.cuda.synchronize()
    assert np.all(step.info.cpu().numpy() == 0), step.info.cpu().numpy()
    M = step.M.double().cpu().numpy()
    nl = len(cfg.lambdas)
    kp = r_prev + cfg.k
    fit = None
    if kp <= 64:  # the realisation error of the fitted adapters (Section S6)
        from paper_2608_03020_amd import loca
        fit = torch.full((len(blocks) * nl * 3,), float("nan"), dtype=torch.float64, device=dev)
        ws = loca.alloc_workspace(loca.workspace_size(loca.LOCA_OP_REALIZATION_ERROR, len(blocks), 0, cfg.d, cfg.k,
                                                      r_a=r_prev, n_lambda=nl), dev)
        ws.fill_(255)
        right = torch.cat([rp_d, B], dim=1).contiguous()
        loca.loca_realization_error(step.M, right, step.K, cfg.lambdas, torch.stack(step.mb_log).contiguous(), fit,
                                    ws, lp=lp_d)
        fit = fit.cpu().numpy().reshape(len(blocks), nl, 3)
    for b in blocks:
        Wp = Lps[b].astype(np.float64) @ Rps[b].astype(np.float64)
        o = oracle.block_step(xf[b], zf, ys, gen.as_f64(As[b], cfg.a_dtype), np.asarray(Bs[b], np.float64), cfg.eta,
                              cfg.lambdas, cfg.r_a, W_prev=Wp)
        right = np.concatenate([Rps[b].astype(np.float64), np.asarray(Bs[b], np.float64)], axis=0)
        for l in range(nl):
            W_ref = o["solves"][l]["W"]
            Wr_ref, sig_ref = oracle.truncate_dense(W_ref, cfg.r_a)
            W_gpu = M[b, l] @ right
            mi = b * nl + l
            Wr_gpu = step.A_ad[mi].double().cpu().numpy().T @ step.B_ad[mi].double().cpu().numpy().T
            sig_gpu = step.sigma[mi].double().cpu().numpy()
            e = {"W": rel(W_gpu, W_ref), "W_r": rel(Wr_gpu, Wr_ref), "sigma": rel(sig_gpu[:cfg.r_a], sig_ref[:cfg.r_a])}
            if fit is not None:
                ref = oracle.realization_error(np.concatenate(xf[b]), np.concatenate(o["T"]), W_ref, Wp)
                e["fit2"] = abs(fit[b, l, 0] - ref["fit2"]) / ref["fit2"]
                e["tar2"] = abs(fit[b, l, 1] - ref["tar2"]) / ref["tar2"]
                e["w2"] = abs(fit[b, l, 2] - ref["w2"]) / ref["w2"]
            log(f"outer_step {mode} block {b} lambda {cfg.lambdas[l]}: " +
                ", ".join(f"{k} {v:.2e}" for k, v in e.items()))
            assert max(e.values()) <= tol, e


@pytest.mark.parametrize("mode", ["bf16", "fp32"])
def test_realization_error_frozen_step_with_weights(mode):
    """Realisation error (Section S6) after the first outer step, with statistic weights
    (20% of positions at a_t = 0): sum_n a_n ||E_fit,n||^2, ||T||^2 and ||W||^2 from the
    factors against the oracle's dense E_fit = X W - T."""
    import torch
    import oracle
    from paper_2608_03020_amd import loca
    from paper_2608_03020_amd.step import BlockStep
    if mode == "bf16":
        cfg = gen.custom_config("t15", blocks=3, d=1040, n=2600, micro=1000, C=5, k=32, r_a=16,
                                lambdas=(1e-3, 1e-1))
        tol = 2e-3
    else:
        cfg = gen.custom_config("t15f", blocks=2, d=180, n=400, micro=150, C=4, k=12, r_a=6, lambdas=(1e-2,),
                                mode="fp32", x_dist="gauss_outlier")
        tol = 1e-5
    nb, nl = cfg.blocks, len(cfg.lambdas)
    log(f"case realisation {mode}: d={cfg.d} n={cfg.n} k={cfg.k} blocks={nb}")
    xs, zs, ys, As, Bs = host_inputs(cfg, range(nb))
    aw = [gen.gen_stat_weights(cfg, m) for m in range(cfg.n_micro)]
    step = BlockStep(cfg, nb, poison=True)
    x_all = padded_rows(np.stack([np.concatenate(xb) for xb in xs]))
    z_all, y_all = to_dev(np.concatenate(zs)), to_dev(np.concatenate(ys))
    a_all = to_dev(np.concatenate(aw))
    A, B = to_dev(np.stack(As)), to_dev(np.stack(Bs))
    step.reset()
    for m in range(cfg.n_micro):
        lo, hi = cfg.micro_rows(m)
        step.micro_batch(x_all[:, lo:hi], z_all[lo:hi], y_all[lo:hi], A, B, keep_log=True, a=a_all[lo:hi])
    step.solve(B)
    fit = torch.full((nb * nl * 3,), float("nan"), dtype=torch.float64, device="cuda")
    ws = loca.alloc_workspace(loca.workspace_size(loca.LOCA_OP_REALIZATION_ERROR, nb, 0, cfg.d, cfg.k,
                                                  n_lambda=nl))
    ws.fill_(255)
    loca.loca_realization_error(step.M, B, step.K, cfg.lambdas, torch.stack(step.mb_log).contiguous(), fit, ws)
    torch.cuda.synchronize()
    assert np.all(step.info.cpu().numpy() == 0)
    fit = fit.cpu().numpy().reshape(nb, nl, 3)
    xmode = "f32" if mode == "fp32" else "bf16"
    for b in range(nb):
        xf = [gen.as_f64(x, xmode) for x in xs[b]]
        o = oracle.block_step(xf, [gen.as_f64(z, cfg.logit_dtype) for z in zs], ys, gen.as_f64(As[b], cfg.a_dtype),
                              np.asarray(Bs[b], np.float64), cfg.eta, cfg.lambdas, cfg.r_a, a_ws=aw)
        for l in range(nl):
            ref = oracle.realization_error(np.concatenate(xf), np.concatenate(o["T"]), o["solves"][l]["W"],
                                           a=np.concatenate(aw))
            e = {q: abs(fit[b, l, i] - ref[q]) / ref[q] for i, q in enumerate(("fit2", "tar2", "w2"))}
            log(f"realisation {mode} block {b} lambda {cfg.lambdas[l]}: fit2/tar2 {ref['fit2'] / ref['tar2']:.3f}, " +
                ", ".join(f"{q} {v:.2e}" for q, v in e.items()))
            assert max(e.values()) <= tol, e


def test_loss_weights_and_masked_positions():
    """Loss weights w_t >= 0 with masked positions (w_t = 0): the head error row is
    w_t (softmax - onehot) (Lemma S3.1 with the weighted sequence loss), so masked
    positions give zero credit coordinates while their rows still enter S and ||X||^2."""
    import torch
    from paper_2608_03020_amd.step import BlockStep
    cfg = gen.custom_config("t15", blocks=2, d=320, n=1100, micro=600, C=5, k=16, r_a=8, lambdas=(1e-2,))
    blocks = [0, 1]
    log(f"case loss_weights: d={cfg.d} n={cfg.n} micro={cfg.micro} C={cfg.C} k={cfg.k}, 20% masked")
    xs, zs, ys, As, Bs = host_inputs(cfg, blocks)
    ws = [gen.gen_loss_weights(cfg, m) for m in range(cfg.n_micro)]
    dev = "cuda"
    step = BlockStep(cfg, len(blocks), dev)
    x_all = padded_rows(np.stack([np.concatenate(xb, axis=0) for xb in xs]), dev)
    z_all, y_all = to_dev(np.concatenate(zs, axis=0), dev), to_dev(np.concatenate(ys, axis=0), dev)
    w_all = to_dev(np.concatenate(ws), dev)
    A, B = to_dev(np.stack(As), dev), to_dev(np.stack(Bs), dev)
    step.reset()
    Ys, mbs = [], []
    for m in range(cfg.n_micro):
        lo, hi = cfg.micro_rows(m)
        step.micro_batch(x_all[:, lo:hi], z_all[lo:hi], y_all[lo:hi], A, B, w=w_all[lo:hi])
        Ys.append(step.Y[:, :hi - lo].double().cpu().numpy())
        mbs.append(step.mb.cpu().numpy().copy())
    step.solve(B)
    torch.cuda.synchronize()
    assert np.all(step.info.cpu().numpy() == 0), step.info.cpu().numpy()
    import oracle
    for b in blocks:
        xf = [gen.as_f64(x, "bf16") for x in xs[b]]
        o = oracle.block_step(xf, [gen.as_f64(z, cfg.logit_dtype) for z in zs], ys, gen.as_f64(As[b], cfg.a_dtype),
                              np.asarray(Bs[b], np.float64), cfg.eta, cfg.lambdas, cfg.r_a,
                              ws=[np.asarray(w, np.float64) for w in ws])
        e = {}
        for m in range(cfg.n_micro):
            e[f"Y{m}"] = rel(Ys[m][b], o["Y"][m])
            masked = ws[m] == 0.0
            assert np.all(Ys[m][b][masked] == 0.0), "masked positions must have zero credit coordinates"
            e[f"q2_{m}"] = abs(mbs[m][b, 0] - o["mb"][m]["sum_q2"]) / o["mb"][m]["sum_q2"]
            e[f"eta{m}"] = abs(mbs[m][b, 2] - o["mb"][m]["eta_bar"]) / o["mb"][m]["eta_bar"]
        iu = np.triu_indices(cfg.d)
        e["S"] = rel(step.S[b].double().cpu().numpy()[iu], o["S"][iu])
        e["K"] = rel(step.K[b].double().cpu().numpy(), o["K"])
        e["M"] = rel(step.M[b, 0].double().cpu().numpy(), o["solves"][0]["M"])
        log(f"loss_weights block {b}: " + ", ".join(f"{k} {v:.2e}" for k, v in e.items()))
        assert max(v for k, v in e.items() if k[0] in "Yqe") <= 1e-5, e
        assert max(e["S"], e["K"], e["M"]) <= 2e-3, e
