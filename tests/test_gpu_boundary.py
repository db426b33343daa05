"""The boundary's device-side reporting and its behaviour under concurrent callers.

* Non-finite data: a NaN or +inf logit, a NaN credit factor or a NaN entry of X is
  reported as LOCA_INFO_NONFINITE in the calling entry point's dev_info; a -inf logit
  is an excluded class (its softmax weight is zero) and is not.
* Every call of a step has its own dev_info slice, so a solve's pivot code is still
  there after the truncation has run.
* Two host threads, each running statistics and then the ridge solve on its own
  stream and buffers, give the bits of the single-threaded runs (the solve's internal
  streams are shared between them).
* The projected solve on the step's side stream, beside the ridge solves, gives the
  bits of the same calls run alone.
"""
import threading

import numpy as np
import pytest

from gpu_helpers import host_inputs, log, padded_rows, to_dev
from paper_2608_03020_amd import inputs as gen

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_03020_amd import loca
    loca.load()


def _error_call(z, y, A, B, n, k, d, C):
    import torch
    from paper_2608_03020_amd import loca
    nb = A.shape[0]
    Y = torch.full((nb, n, k), float("nan"), device="cuda")
    mb = loca.new_mb(nb)
    info = torch.full((1,), 12345, dtype=torch.int32, device="cuda")
    ws = loca.alloc_workspace(loca.workspace_size(loca.LOCA_OP_ERROR_TARGETS, nb, n, d, k, C))
    loca.loca_error_targets(z, y, A, B, Y, mb, info, ws)
    torch.cuda.synchronize()
    return int(info.item()), Y, mb


@pytest.mark.parametrize("C,ldt,adt", [(5, "f32", "f32"), (3001, "bf16", "bf16"), (3001, "f32", "f32")])
def test_nonfinite_logits_reported(C, ldt, adt):
    """Small label set, the vocabulary product (bf16 A~) and the streaming kernel (fp32 A~)."""
    import torch
    from paper_2608_03020_amd import loca
    n, k, d, nb = 300, 16, 64, 2
    log(f"case non-finite logits C={C} logits {ldt} A~ {adt}")
    g = torch.Generator(device="cuda")
    g.manual_seed(5)
    zt = torch.bfloat16 if ldt == "bf16" else torch.float32
    at = torch.bfloat16 if adt == "bf16" else torch.float32
    ld = (C + 7) // 8 * 8  # 16-byte rows: the vocabulary product reads them in 16-byte chunks
    z0_buf = torch.zeros((n, ld), device="cuda", dtype=zt)
    z0_buf[:, :C] = (torch.randn((n, C), generator=g, device="cuda") * 2).to(zt)
    y = torch.randint(0, C, (n,), generator=g, device="cuda", dtype=torch.int32)

    class _Z:  # logits rows of stride ld; clone() keeps the stride
        def __init__(self, buf):
            self.buf = buf

        def clone(self):
            return _Z(self.buf.clone())

        def __setitem__(self, ij, v):
            self.buf[ij] = v

        @property
        def view(self):
            return self.buf[:, :C]
    z0 = _Z(z0_buf)
    A = (torch.randn((nb, C, k), generator=g, device="cuda") / np.sqrt(k)).to(at)
    B = torch.randn((nb, k, d), generator=g, device="cuda") / np.sqrt(k)

    code, Y, _ = _error_call(z0.view, y, A, B, n, k, d, C)
    assert code == 0 and not bool(torch.isnan(Y).any())
    # -inf logit (not the label): an excluded class, the call is fine
    z = z0.clone()
    col = (int(y[7].item()) + 1) % C
    z[7, col] = float("-inf")  # a class other than the label
    code, Y, _ = _error_call(z.view, y, A, B, n, k, d, C)
    assert code == 0 and bool(torch.isfinite(Y).all())
    for bad in (float("nan"), float("inf")):
        z = z0.clone()
        z[211, 2] = bad
        code, _, _ = _error_call(z.view, y, A, B, n, k, d, C)
        assert code == loca.LOCA_INFO_NONFINITE, (bad, code)
    # a non-finite value takes precedence over an out-of-range label
    z = z0.clone()
    z[5, 0] = float("nan")
    y2 = y.clone()
    y2[3] = C + 4
    code, _, _ = _error_call(z.view, y2, A, B, n, k, d, C)
    assert code == loca.LOCA_INFO_NONFINITE
    # a NaN in one block's credit factor
    A2 = A.clone()
    A2[1, 0, 0] = float("nan")
    code, _, _ = _error_call(z0.view, y, A2, B, n, k, d, C)
    assert code == loca.LOCA_INFO_NONFINITE


def test_nonfinite_top_error_reported():
    import torch
    from paper_2608_03020_amd import loca
    n, V, d = 64, 1000, 64
    g = torch.Generator(device="cuda")
    g.manual_seed(6)
    z = torch.randn((n, V), generator=g, device="cuda").to(torch.bfloat16)
    y = torch.randint(0, V, (n,), generator=g, device="cuda", dtype=torch.int32)
    Wu = (torch.randn((V, d), generator=g, device="cuda") / 8).to(torch.bfloat16)
    e = torch.empty((n, d), device="cuda")
    info = torch.full((1,), 7, dtype=torch.int32, device="cuda")
    ws = loca.alloc_workspace(loca.workspace_size(loca.LOCA_OP_TOP_ERROR, 1, n, d, 1, V))
    loca.loca_top_error(z, y, Wu, e, info, ws)
    torch.cuda.synchronize()
    assert info.item() == 0
    z[9, 17] = float("nan")
    loca.loca_top_error(z, y, Wu, e, info, ws)
    torch.cuda.synchronize()
    assert info.item() == loca.LOCA_INFO_NONFINITE


@pytest.mark.parametrize("mode", ["bf16", "fp32"])
def test_nonfinite_x_reported(mode):
    """A NaN entry of one block's X is reported for that block only."""
    import torch
    from paper_2608_03020_amd.step import BlockStep
    cfg = gen.custom_config("nf", blocks=3, d=1040 if mode == "bf16" else 200, n=700, micro=700, C=5, k=16,
                            r_a=4, mode=mode, x_dist="gauss_outlier" if mode == "fp32" else "rms_outlier",
                            logit_dtype="f32")
    log(f"case non-finite X, {mode}")
    xs, zs, ys, As, Bs = host_inputs(cfg, range(3))
    x_all = padded_rows(np.stack([np.concatenate(xb) for xb in xs]))
    z_all, y_all = to_dev(np.concatenate(zs)), to_dev(np.concatenate(ys))
    A, B = to_dev(np.stack(As)), to_dev(np.stack(Bs))
    st = BlockStep(cfg, 3)
    st.reset()
    st.micro_batch(x_all, z_all, y_all, A, B)
    torch.cuda.synchronize()
    assert np.all(st.info_stats.cpu().numpy() == 0)
    x_bad = x_all.clone()
    x_bad[1, 333, 17] = float("nan")
    st.reset()
    st.micro_batch(x_bad, z_all, y_all, A, B)
    torch.cuda.synchronize()
    assert st.info_stats.cpu().numpy()[0].tolist() == [0, -1, 0]
    assert int(st.info_err[0].item()) == 0


def test_solve_pivot_code_survives_the_step():
    """An indefinite S (overwritten after the statistics) makes the solve report its first
    pivot; the truncation that follows has its own slice and does not erase the code."""
    import torch
    from paper_2608_03020_amd.step import BlockStep
    cfg = gen.custom_config("piv", blocks=3, d=300, n=800, micro=400, C=5, k=8, r_a=4)
    xs, zs, ys, As, Bs = host_inputs(cfg, range(3))
    x_all = padded_rows(np.stack([np.concatenate(xb) for xb in xs]))
    z_all, y_all = to_dev(np.concatenate(zs)), to_dev(np.concatenate(ys))
    A, B = to_dev(np.stack(As)), to_dev(np.stack(Bs))
    st = BlockStep(cfg, 3)
    st.reset()
    for m in range(cfg.n_micro):
        lo, hi = cfg.micro_rows(m)
        st.micro_batch(x_all[:, lo:hi], z_all[lo:hi], y_all[lo:hi], A, B)
    st.S[2].copy_(-torch.eye(cfg.d, device="cuda"))  # indefinite: the first pivot fails
    st.solve(B)
    torch.cuda.synchronize()
    assert st.info_solve.cpu().numpy().tolist() == [0, 0, 1]
    assert np.all(st.info_trunc.cpu().numpy() == 0)
    assert np.all(st.info_err.cpu().numpy() == 0) and np.all(st.info_stats.cpu().numpy() == 0)
    info = st.info.cpu().numpy()
    assert np.count_nonzero(info) == 1


def test_concurrent_solves_from_two_threads():
    """Two host threads, each on its own stream with its own buffers, run the statistics
    and then the ridge solve (three blocks: the solve uses its internal streams) several
    times; every result equals, bit for bit, the same work run alone."""
    import torch
    from paper_2608_03020_amd.step import BlockStep
    cfg = gen.custom_config("thr", blocks=3, d=1024, n=2048, micro=1024, C=5, k=16, r_a=8, lambdas=(1e-2, 1e-1))
    inputs = []
    for seed in (1, 2):
        xs, zs, ys, As, Bs = host_inputs(cfg, range(3), seed=seed)
        inputs.append((padded_rows(np.stack([np.concatenate(xb) for xb in xs])), to_dev(np.concatenate(zs)),
                       to_dev(np.concatenate(ys)), to_dev(np.stack(As)), to_dev(np.stack(Bs))))

    def work(i, st):
        x_all, z_all, y_all, A, B = inputs[i]
        st.run(x_all, z_all, y_all, A, B)

    ref = []
    for i in range(2):
        st = BlockStep(cfg, 3)
        work(i, st)
        torch.cuda.synchronize()
        ref.append((st.S.cpu().numpy(), st.K.cpu().numpy(), st.M.cpu().numpy(), st.sigma.cpu().numpy()))
    log("case two threads: references done")
    reps = 4
    steps = [[BlockStep(cfg, 3) for _ in range(reps)] for _ in range(2)]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]  # default priority
    errors = []

    def thread_main(i):
        try:
            with torch.cuda.stream(streams[i]):
                for r in range(reps):
                    work(i, steps[i][r])
        except Exception as ex:  # reported in the main thread
            errors.append(ex)

    ths = [threading.Thread(target=thread_main, args=(i,)) for i in range(2)]
    for t in ths:
        t.start()
    for t in ths:
        t.join()
    torch.cuda.synchronize()
    assert not errors, errors
    for i in range(2):
        for r in range(reps):
            st = steps[i][r]
            got = (st.S.cpu().numpy(), st.K.cpu().numpy(), st.M.cpu().numpy(), st.sigma.cpu().numpy())
            for a, b in zip(got, ref[i]):
                assert np.array_equal(a, b), (i, r)
            assert np.all(st.info.cpu().numpy() == 0)


def test_projected_solve_beside_ridge_solves():
    """The projected solve runs on the step's side stream beside the ridge solves (three
    blocks, so the solves use their internal streams too); over three steps in a row M,
    the truncation and B* equal, bit for bit, the ridge solve run alone and the projected
    solve called alone on the same statistics."""
    import torch
    from paper_2608_03020_amd import loca
    from paper_2608_03020_amd.step import BlockStep
    cfg = gen.custom_config("side", blocks=3, d=1024, n=2048, micro=1024, C=5, k=16, r_a=8, lambdas=(1e-2, 1e-1))
    xs, zs, ys, As, Bs = host_inputs(cfg, range(3), seed=3)
    x_all = padded_rows(np.stack([np.concatenate(xb) for xb in xs]))
    z_all, y_all = to_dev(np.concatenate(zs)), to_dev(np.concatenate(ys))
    A, B = to_dev(np.stack(As)), to_dev(np.stack(Bs))
    proj = gen.torch_gen_adapter_projection(cfg, 3)
    log("case projected solve on the side stream: 3 blocks, 2 lambdas, 3 steps")
    ref = BlockStep(cfg, 3)
    ref.run(x_all, z_all, y_all, A, B)
    nl = len(cfg.lambdas)
    b_ref = torch.empty((3, nl, cfg.d, cfg.r_a), device="cuda")
    info_ref = torch.zeros(3 * nl, dtype=torch.int32, device="cuda")
    ws = loca.alloc_workspace(loca.workspace_size(loca.LOCA_OP_RIDGE_SOLVE_PROJECTED, 3, cfg.micro, cfg.d, cfg.k,
                                                  cfg.C, cfg.r_a, nl, ref.acc))
    loca.loca_ridge_solve_projected(ref.S, ref.K, B, proj, cfg.lambdas, b_ref, info_ref, ws)
    torch.cuda.synchronize()
    st = BlockStep(cfg, 3, projected=True, poison=True)
    for rep in range(3):
        st.B_proj.fill_(float("nan"))
        st.run(x_all, z_all, y_all, A, B, proj_a=proj)
        torch.cuda.synchronize()
        assert np.array_equal(st.M.cpu().numpy(), ref.M.cpu().numpy()), rep
        assert np.array_equal(st.sigma.cpu().numpy(), ref.sigma.cpu().numpy()), rep
        assert np.array_equal(st.B_proj.cpu().numpy(), b_ref.cpu().numpy()), rep
        assert np.all(st.info.cpu().numpy() == 0) and np.all(info_ref.cpu().numpy() == 0)
