"""C-ABI checks that need no GPU: the library loads, exports every entry point
declared in include/loca.h, and rejects invalid arguments synchronously
(before anything is enqueued, so no device is touched)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "loca.h")


@pytest.fixture(scope="module")
def lib():
    from paper_2608_03020_amd import loca
    if not os.path.exists(loca.LIB_PATH):
        pytest.skip("libloca.so not built (run __graft_entry__.build())")
    return loca


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(loca_[a-z_]+)\s*\(", text)))


def test_header_declares_the_four_step_calls():
    names = declared_functions()
    for fn in ("loca_error_targets", "loca_accumulate_stats", "loca_ridge_solve", "loca_lowrank_truncate"):
        assert fn in names


def test_every_declared_symbol_is_exported(lib):
    so = ctypes.CDLL(lib.LIB_PATH)
    for name in declared_functions():
        assert hasattr(so, name), name
    assert set(lib.EXPORTED) == set(declared_functions())


def test_status_strings_and_version(lib):
    assert lib.status_str(lib.LOCA_OK) == "ok"
    assert "argument" in lib.status_str(lib.LOCA_E_ARG)
    assert "gfx950" in lib.version()


def test_workspace_sizes_are_positive_and_monotone(lib):
    a = lib.workspace_size(lib.LOCA_OP_ACCUMULATE_STATS, 1, 512, 896, 8, acc=lib.LOCA_F64)
    b = lib.workspace_size(lib.LOCA_OP_ACCUMULATE_STATS, 2, 512, 896, 8, acc=lib.LOCA_F64)
    assert 0 < a < b
    s1 = lib.workspace_size(lib.LOCA_OP_RIDGE_SOLVE, 1, 0, 1536, 16, n_lambda=1)
    s3 = lib.workspace_size(lib.LOCA_OP_RIDGE_SOLVE, 1, 0, 1536, 16, n_lambda=3)
    assert s3 > s1 >= 4 * 1536 * 1536
    assert lib.workspace_size(lib.LOCA_OP_ERROR_TARGETS, 0, 10, 10, 4) == 0


FAKE = 0x100000  # never dereferenced: every call below fails validation first


def test_error_targets_rejects(lib):
    so = lib.load()
    ok_args = dict(stream=None, nb=1, n=8, C=4, k=2, d=16, logits=FAKE, ldt=lib.LOCA_F32, ld=4, labels=FAKE, w=None,
                   aw=None, a=FAKE, adt=lib.LOCA_F32, abs_=0, b=FAKE, bbs=0, y=FAKE, ybs=0, e=None, mb=FAKE, info=FAKE,
                   ws=None, wsb=0)

    def call(**kw):
        a = dict(ok_args, **kw)
        return so.loca_error_targets(a["stream"], a["nb"], a["n"], a["C"], a["k"], a["d"], a["logits"], a["ldt"],
                                     a["ld"], a["labels"], a["w"], a["aw"], a["a"], a["adt"], a["abs_"], a["b"], a["bbs"],
                                     None, a["y"], a["ybs"], a["e"], a["mb"], a["info"], a["ws"], a["wsb"])

    assert call(n=0) == lib.LOCA_E_ARG
    assert call(C=0) == lib.LOCA_E_ARG
    assert call(logits=None) == lib.LOCA_E_ARG
    assert call(ld=3) == lib.LOCA_E_ARG
    assert call(ldt=lib.LOCA_F64) == lib.LOCA_E_ARG
    assert call(nb=2, abs_=1) == lib.LOCA_E_ARG
    assert call(k=129) == lib.LOCA_E_UNSUPPORTED
    assert call() == lib.LOCA_E_WORKSPACE                  # missing workspace
    assert call(ws=FAKE + 1, wsb=1 << 30) == lib.LOCA_E_WORKSPACE  # misaligned


def test_error_targets_noalloc_rejects(lib):
    """Argument errors and sizes whose workspace exceeds the fixed scratch array are
    reported before the array is looked up on a device."""
    so = lib.load()

    def call(nb=1, n=8, C=4, k=2, d=16, logits=FAKE, info=FAKE):
        return so.loca_error_targets_noalloc(None, nb, n, C, k, d, logits, lib.LOCA_F32, C, FAKE, None, None, FAKE,
                                             lib.LOCA_F32, 0, FAKE, 0, None, FAKE, 0, None, FAKE, info)

    assert call(n=0) == lib.LOCA_E_ARG
    assert call(logits=None) == lib.LOCA_E_ARG
    assert call(info=None) == lib.LOCA_E_ARG
    assert call(k=129) == lib.LOCA_E_UNSUPPORTED
    assert call(n=4096, C=151936, k=64, d=2048) == lib.LOCA_E_UNSUPPORTED   # ~34 MB of scratch
    assert lib.error_targets_noalloc_max_bytes() == 16 << 20
    big = lib.workspace_size(lib.LOCA_OP_ERROR_TARGETS, 48, 65536, 5120, 64, 5)
    assert big <= lib.error_targets_noalloc_max_bytes()  # the largest small-label workload fits


def test_credit_gram_rejects_and_layout(lib):
    so = lib.load()
    assert [lib.credit_gram_ld(k) for k in (1, 16, 17, 32, 33, 64, 65, 128)] == [16, 16, 32, 32, 64, 64, 65, 128]
    assert so.loca_credit_gram(None, 1, 0, 16, FAKE, 0, FAKE, None, 0) == lib.LOCA_E_ARG
    assert so.loca_credit_gram(None, 1, 4, 16, None, 0, FAKE, None, 0) == lib.LOCA_E_ARG
    assert so.loca_credit_gram(None, 2, 4, 16, FAKE, 8, FAKE, None, 0) == lib.LOCA_E_ARG   # block stride < k d
    assert so.loca_credit_gram(None, 1, 129, 16, FAKE, 0, FAKE, None, 0) == lib.LOCA_E_UNSUPPORTED
    assert so.loca_credit_gram(None, 1, 4, 16, FAKE, 0, FAKE, None, 0) == lib.LOCA_E_WORKSPACE


def test_accumulate_stats_rejects(lib):
    so = lib.load()
    base = [None, 1, 64, 32, 4, FAKE, lib.LOCA_BF16, 32, 0, FAKE, 0, None, 0.01, FAKE, FAKE, FAKE, lib.LOCA_F32,
            0, 0, 1, None, None, 0]

    def call(**kw):
        idx = dict(nb=1, n=2, d=3, k=4, x=5, xdt=6, ldx=7, xbs=8, eta=12, S=14, acc=16)
        a = list(base)
        for key, v in kw.items():
            a[idx[key]] = v
        return so.loca_accumulate_stats(*a)

    assert call(d=0) == lib.LOCA_E_ARG
    assert call(ldx=31) == lib.LOCA_E_ARG
    assert call(ldx=36) == lib.LOCA_E_ARG                  # bf16 rows must be 16-byte multiples
    assert call(x=FAKE + 2) == lib.LOCA_E_ARG              # misaligned base
    assert call(eta=-1.0) == lib.LOCA_E_ARG
    assert call(eta=float("nan")) == lib.LOCA_E_ARG
    assert call(acc=lib.LOCA_F64) == lib.LOCA_E_ARG        # bf16 X needs fp32 statistics
    assert call(xdt=lib.LOCA_F32) == lib.LOCA_E_ARG        # fp32 X needs fp64 statistics
    assert call(S=None) == lib.LOCA_E_ARG
    assert call(nb=2, xbs=10) == lib.LOCA_E_ARG
    assert call(k=200) == lib.LOCA_E_UNSUPPORTED
    assert call() == lib.LOCA_E_WORKSPACE


def _lams(*v):
    arr = (ctypes.c_double * len(v))(*v)
    return ctypes.cast(arr, ctypes.c_void_p), arr


def test_ridge_solve_rejects(lib):
    so = lib.load()

    def call(lams=(1e-2,), d=16, k=4, acc=lib.LOCA_F32, S=FAKE, r_prev=0, lp=None, mbs=64, ws=None):
        p, _keep = _lams(*lams) if lams is not None else (None, None)
        return so.loca_ridge_solve(None, 1, d, k, S, FAKE, acc, 0, 0, lp, None, r_prev, 0, 0, p,
                                   len(lams) if lams else 0, FAKE, mbs, None, 0, None, 0, FAKE, ws, 0)

    assert call(lams=(0.0,)) == lib.LOCA_E_ARG            # the paper requires lambda > 0
    assert call(lams=(1e-2, -1.0)) == lib.LOCA_E_ARG
    assert call(lams=(float("inf"),)) == lib.LOCA_E_ARG
    assert call(lams=None) == lib.LOCA_E_ARG
    assert call(acc=lib.LOCA_BF16) == lib.LOCA_E_ARG
    assert call(S=None) == lib.LOCA_E_ARG
    assert call(r_prev=2, lp=None) == lib.LOCA_E_ARG
    assert call(k=129) == lib.LOCA_E_UNSUPPORTED
    assert call(lams=tuple([0.1] * 9)) == lib.LOCA_E_UNSUPPORTED
    assert call() == lib.LOCA_E_WORKSPACE


def test_lowrank_truncate_rejects(lib):
    so = lib.load()

    def call(d=32, kp=8, r_a=4, r_group=1, m=FAKE):
        return so.loca_lowrank_truncate(None, 1, d, kp, r_a, m, 0, FAKE, 0, r_group, FAKE, 0, FAKE, 0, FAKE, 0,
                                        None, 0, FAKE, None, 0)

    assert call(r_a=9) == lib.LOCA_E_ARG                   # r_a <= kp
    assert call(kp=40, r_a=4) == lib.LOCA_E_ARG            # kp <= d
    assert call(r_group=0) == lib.LOCA_E_ARG
    assert call(m=None) == lib.LOCA_E_ARG
    assert call(d=200, kp=129, r_a=4) == lib.LOCA_E_UNSUPPORTED  # kp <= 128
    assert call(d=200, kp=100, r_a=65) == lib.LOCA_E_UNSUPPORTED  # r_a <= 64
    assert call(d=100, kp=65, r_a=4) == lib.LOCA_E_WORKSPACE     # supported: only the workspace is missing
    assert call() == lib.LOCA_E_WORKSPACE


def test_projected_and_dense_targets_reject(lib):
    so = lib.load()
    p, _keep = _lams(1e-2)
    assert so.loca_ridge_solve_projected(None, 1, 16, 4, 0, FAKE, FAKE, lib.LOCA_F32, 0, 0, FAKE, 0, FAKE, 0, None,
                                         0, p, 1, FAKE, 0, None, FAKE, None, 0) == lib.LOCA_E_ARG
    assert so.loca_ridge_solve_projected(None, 1, 16, 4, 65, FAKE, FAKE, lib.LOCA_F32, 0, 0, FAKE, 0, FAKE, 0, None,
                                         0, p, 1, FAKE, 0, None, FAKE, None, 0) == lib.LOCA_E_UNSUPPORTED
    assert so.loca_dense_targets(None, 1, 4, 2, 8, None, 0, FAKE, FAKE, 0, FAKE, 0) == lib.LOCA_E_ARG


def test_feedback_fit_rejects(lib):
    so = lib.load()

    def call(nb=1, d=32, n_p=16, k=4, e=FAKE, g=FAKE, gbs=0, beta=0.1, wu=None, wdt=lib.LOCA_F32, vocab=0,
             bt=FAKE, at=None, vk=None, vkbs=0, sig=FAKE, alpha=FAKE, ws=None, wsb=0):
        return so.loca_feedback_fit(None, nb, d, n_p, k, e, g, gbs, beta, wu, wdt, vocab, bt, 0, at, 0, vk, vkbs, sig,
                                    alpha, FAKE, ws, wsb)

    assert call(beta=0.0) == lib.LOCA_E_ARG               # the fit needs beta > 0
    assert call(beta=float("inf")) == lib.LOCA_E_ARG
    assert call(beta=float("nan")) == lib.LOCA_E_ARG
    assert call(k=17) == lib.LOCA_E_ARG                   # k <= np
    assert call(d=3) == lib.LOCA_E_ARG                    # k <= d
    assert call(e=None) == lib.LOCA_E_ARG
    assert call(at=FAKE) == lib.LOCA_E_ARG                # A~ needs W_u
    assert call(at=FAKE, wu=FAKE, vocab=10, wdt=lib.LOCA_F64) == lib.LOCA_E_ARG
    assert call(nb=2, gbs=10) == lib.LOCA_E_ARG
    assert call(nb=2, gbs=32 * 16, vk=FAKE, vkbs=10) == lib.LOCA_E_ARG  # V_k stride below d k
    assert call(n_p=65, k=4) == lib.LOCA_E_UNSUPPORTED
    assert call(d=8, n_p=16, k=4) == lib.LOCA_E_UNSUPPORTED  # np <= d
    assert call() == lib.LOCA_E_WORKSPACE
    assert so.loca_workspace_size(lib.LOCA_OP_FEEDBACK_FIT, 2, 48, 300, 8, 0, 0, 0, lib.LOCA_F32) > 0
    assert so.loca_workspace_size(lib.LOCA_OP_FEEDBACK_FIT, 2, 65, 300, 8, 0, 0, 0, lib.LOCA_F32) == 0


def test_feedback_fit_primal_rejects(lib):
    so = lib.load()

    def call(nb=1, d=256, n_p=100, k=8, beta=0.1, ws=None, wsb=0):
        return so.loca_feedback_fit_primal(None, nb, d, n_p, k, FAKE, FAKE, 0, beta, None, lib.LOCA_F32, 0, FAKE, 0,
                                           None, 0, None, 0, FAKE, FAKE, FAKE, ws, wsb)

    assert call(beta=0.0) == lib.LOCA_E_ARG
    assert call(k=101) == lib.LOCA_E_ARG                  # k <= np
    assert call(n_p=129) == lib.LOCA_E_UNSUPPORTED        # np <= 128
    assert call(n_p=100, k=65) == lib.LOCA_E_UNSUPPORTED  # k <= 64 (the truncation's rank limit)
    assert call(d=90) == lib.LOCA_E_UNSUPPORTED           # np <= d
    assert call(d=70000) == lib.LOCA_E_UNSUPPORTED        # the d x d solve's limit
    assert call() == lib.LOCA_E_WORKSPACE
    need = so.loca_workspace_size(lib.LOCA_OP_FEEDBACK_FIT_PRIMAL, 1, 100, 256, 8, 0, 0, 0, lib.LOCA_F32)
    assert need >= 8 * 256 * 256                          # holds E E^T in float64
    assert call(ws=FAKE, wsb=need - 1) == lib.LOCA_E_WORKSPACE
    assert so.loca_workspace_size(lib.LOCA_OP_FEEDBACK_FIT_PRIMAL, 1, 129, 256, 8, 0, 0, 0, lib.LOCA_F32) == 0


def test_feedback_fit_large_rejects(lib):
    so = lib.load()

    def call(nb=1, d=256, n_p=600, k=8, l=32, q=3, om=FAKE, beta=0.1, ws=None, wsb=0):
        return so.loca_feedback_fit_large(None, nb, d, n_p, k, l, q, FAKE, FAKE, 0, om, beta, None, lib.LOCA_F32, 0,
                                          FAKE, 0, None, 0, None, 0, FAKE, FAKE, FAKE, ws, wsb)

    assert call(beta=0.0) == lib.LOCA_E_ARG
    assert call(om=None) == lib.LOCA_E_ARG                 # the start block is the caller's
    assert call(q=-1) == lib.LOCA_E_ARG
    assert call(k=33) == lib.LOCA_E_ARG                    # k <= l
    assert call(d=30, l=32) == lib.LOCA_E_ARG              # l <= d
    assert call(l=129, d=256) == lib.LOCA_E_UNSUPPORTED    # l <= 128
    assert call(k=65, l=100) == lib.LOCA_E_UNSUPPORTED     # k <= 64
    assert call(q=65) == lib.LOCA_E_UNSUPPORTED
    assert call() == lib.LOCA_E_WORKSPACE
    need = so.loca_workspace_size(lib.LOCA_OP_FEEDBACK_FIT_LARGE, 1, 600, 256, 8, 0, 32, 0, lib.LOCA_F32)
    assert need >= 8 * 256 * 256 + 4 * 256 * 600          # E E^T (float64) and R^T (float)
    assert call(ws=FAKE, wsb=need - 1) == lib.LOCA_E_WORKSPACE
    assert so.loca_workspace_size(lib.LOCA_OP_FEEDBACK_FIT_LARGE, 1, 600, 256, 8, 0, 0, 0, lib.LOCA_F32) == 0


def test_fused_head_rejects(lib):
    so = lib.load()

    def call(n=10, V=100, d=64, c=8, h=FAKE, ldh=64, wu=FAKE, y=FAKE, vm=FAKE, ldvm=8, out=FAKE, ldo=8, ws=None,
             wsb=0):
        return so.loca_fused_head(None, n, V, d, c, h, ldh, wu, y, None, vm, ldvm, out, ldo, FAKE, ws, wsb)

    assert call(h=None) == lib.LOCA_E_ARG
    assert call(ldh=60) == lib.LOCA_E_ARG                 # ldh >= d
    assert call(ldh=68) == lib.LOCA_E_ARG                 # ldh % 8 == 0 (16-byte rows)
    assert call(h=FAKE + 2) == lib.LOCA_E_ARG             # 16-byte aligned h
    assert call(ldvm=4) == lib.LOCA_E_ARG
    assert call(ldo=4) == lib.LOCA_E_ARG
    assert call(d=60, ldh=64) == lib.LOCA_E_UNSUPPORTED   # d % 8 == 0
    assert call() == lib.LOCA_E_WORKSPACE
    need = so.loca_workspace_size(lib.LOCA_OP_FUSED_HEAD, 1, 10, 64, 8, 100, 0, 0, lib.LOCA_F32)
    assert need >= 2 * 8 * 128                            # holds Vm^T padded to whole vocabulary chunks
    assert call(ws=FAKE, wsb=need - 1) == lib.LOCA_E_WORKSPACE


def test_top_error_rejects(lib):
    so = lib.load()

    def call(n=16, V=100, d=64, z=FAKE, zdt=lib.LOCA_BF16, ld=104, y=FAKE, w=None, wu=FAKE, wdt=lib.LOCA_BF16,
             e=FAKE, lde=64, info=FAKE, ws=None, wsb=0):
        return so.loca_top_error(None, n, V, d, z, zdt, ld, y, w, wu, wdt, e, lde, info, ws, wsb)

    assert call(n=0) == lib.LOCA_E_ARG
    assert call(z=None) == lib.LOCA_E_ARG
    assert call(ld=99) == lib.LOCA_E_ARG                   # ld_logits >= V
    assert call(ld=101) == lib.LOCA_E_ARG                  # bf16 rows in 16-byte multiples
    assert call(lde=63) == lib.LOCA_E_ARG
    assert call(z=FAKE + 2) == lib.LOCA_E_ARG              # misaligned logits
    assert call(zdt=lib.LOCA_F64) == lib.LOCA_E_ARG
    assert call(wdt=lib.LOCA_F32) == lib.LOCA_E_UNSUPPORTED  # W_u enters the matrix cores as bf16
    assert call(d=60, lde=64) == lib.LOCA_E_UNSUPPORTED    # d % 8 == 0
    assert call() == lib.LOCA_E_WORKSPACE
    assert so.loca_workspace_size(lib.LOCA_OP_TOP_ERROR, 1, 16, 64, 1, 100, 0, 0, lib.LOCA_F32) > 0


def test_credit_from_top_error_rejects(lib):
    so = lib.load()

    def call(nb=1, n=16, d=64, k=8, e=FAKE, lde=64, v=FAKE, vbs=0, b=FAKE, bbs=0, aw=None, y=FAKE, ybs=0, mb=FAKE,
             ws=None, wsb=0):
        return so.loca_credit_from_top_error(None, nb, n, d, k, e, lde, v, vbs, b, bbs, aw, y, ybs, mb, ws, wsb)

    assert call(k=0) == lib.LOCA_E_ARG
    assert call(v=None) == lib.LOCA_E_ARG
    assert call(lde=32) == lib.LOCA_E_ARG
    assert call(nb=2, vbs=64 * 8 - 1, bbs=8 * 64, ybs=16 * 8) == lib.LOCA_E_ARG
    assert call(k=129) == lib.LOCA_E_UNSUPPORTED
    assert call() == lib.LOCA_E_WORKSPACE
    assert so.loca_workspace_size(lib.LOCA_OP_CREDIT_FROM_TOP_ERROR, 3, 16, 64, 8, 0, 0, 0, lib.LOCA_F32) > 0


def test_binding_rejects_layouts_the_abi_cannot_describe(lib):
    """Arrays the C ABI takes without a row stride must have packed rows; a transposed or
    column-sliced tensor raises in the binding instead of being read with wrong strides."""
    import torch
    with pytest.raises(ValueError):
        lib._ptr(torch.zeros(8, 96).T)                    # rows not contiguous
    with pytest.raises(ValueError):
        lib._ptr(torch.zeros(3, 8, 96).transpose(1, 2))   # block of a transposed stack
    with pytest.raises(ValueError):
        lib._ptr(torch.zeros(10, 16)[:, :8])              # rows not packed
    assert lib._ptr(torch.zeros(10, 16)[:, :8], False) is not None  # arrays with a leading dimension
    assert lib._ptr(torch.zeros(10, 16)[2:5]) is not None
    assert lib._ptr(torch.zeros(4, 1, 3)) is not None
