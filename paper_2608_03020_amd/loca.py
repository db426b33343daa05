"""Thin ctypes binding of libloca (include/loca.h).

Argument marshalling only: every step runs in the library's HIP kernels.
Tensors are torch device tensors; the stream is torch's current stream unless
given.  Each function has the name of the C entry point it calls.  A missing
library raises: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.environ.get("LOCA_LIB", os.path.join(HERE, "lib", "libloca.so"))

LOCA_OK, LOCA_E_ARG, LOCA_E_WORKSPACE, LOCA_E_HIP, LOCA_E_UNSUPPORTED = range(5)
LOCA_F32, LOCA_BF16, LOCA_F64 = range(3)
LOCA_INFO_NONFINITE = -1
LOCA_INFO_BASIS_RANK = -2
(LOCA_OP_ERROR_TARGETS, LOCA_OP_ACCUMULATE_STATS, LOCA_OP_RIDGE_SOLVE, LOCA_OP_LOWRANK_TRUNCATE,
 LOCA_OP_RIDGE_SOLVE_PROJECTED, LOCA_OP_FEEDBACK_FIT, LOCA_OP_TOP_ERROR, LOCA_OP_CREDIT_FROM_TOP_ERROR,
 LOCA_OP_REALIZATION_ERROR, LOCA_OP_CREDIT_GRAM, LOCA_OP_FEEDBACK_FIT_PRIMAL, LOCA_OP_FEEDBACK_FIT_LARGE,
 LOCA_OP_FUSED_HEAD) = range(13)

ENTRY_POINTS = ("loca_error_targets", "loca_accumulate_stats", "loca_ridge_solve", "loca_lowrank_truncate",
                "loca_ridge_solve_projected", "loca_dense_targets", "loca_feedback_fit", "loca_top_error",
                "loca_credit_from_top_error", "loca_error_targets_noalloc", "loca_realization_error",
                "loca_credit_gram", "loca_feedback_fit_primal", "loca_feedback_fit_large", "loca_fused_head")
EXPORTED = ENTRY_POINTS + ("loca_workspace_size", "loca_status_str", "loca_version",
                           "loca_error_targets_noalloc_max_bytes", "loca_credit_gram_ld")


class LocaMB(ctypes.Structure):
    _fields_ = [("sum_q2", ctypes.c_double), ("sum_x2", ctypes.c_double), ("eta_bar", ctypes.c_double),
                ("n", ctypes.c_int64)]


MB_BYTES = ctypes.sizeof(LocaMB)  # 32


class LocaError(RuntimeError):
    def __init__(self, fn: str, status: int):
        self.status = status
        super().__init__(f"{fn} failed: {status_str(status)} ({status})")


_lib = None
_VP, _I64, _SZ, _D = ctypes.c_void_p, ctypes.c_int64, ctypes.c_size_t, ctypes.c_double
_I = ctypes.c_int


def load():
    """Load libloca.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"libloca is not built ({LIB_PATH}); run paper_2608_03020_amd/build.py")
    lib = ctypes.CDLL(LIB_PATH)
    lib.loca_error_targets.argtypes = [_VP, _I64, _I64, _I64, _I64, _I64, _VP, _I, _I64, _VP, _VP, _VP, _VP, _I,
                                       _I64, _VP, _I64, _VP, _VP, _I64, _VP, _VP, _VP, _VP, _SZ]
    lib.loca_error_targets_noalloc.argtypes = [_VP, _I64, _I64, _I64, _I64, _I64, _VP, _I, _I64, _VP, _VP, _VP, _VP,
                                               _I, _I64, _VP, _I64, _VP, _VP, _I64, _VP, _VP, _VP]
    lib.loca_credit_gram.argtypes = [_VP, _I64, _I64, _I64, _VP, _I64, _VP, _VP, _SZ]
    lib.loca_credit_gram_ld.argtypes = [_I64]
    lib.loca_credit_gram_ld.restype = _I64
    lib.loca_error_targets_noalloc_max_bytes.argtypes = []
    lib.loca_error_targets_noalloc_max_bytes.restype = _SZ
    lib.loca_accumulate_stats.argtypes = [_VP, _I64, _I64, _I64, _I64, _VP, _I, _I64, _I64, _VP, _I64, _VP, _D,
                                          _VP, _VP, _VP, _I, _I64, _I64, _I, _VP, _VP, _SZ]
    lib.loca_ridge_solve.argtypes = [_VP, _I64, _I64, _I64, _VP, _VP, _I, _I64, _I64, _VP, _VP, _I64, _I64, _I64,
                                     _VP, _I64, _VP, _I64, _VP, _I64, _VP, _I64, _VP, _VP, _SZ]
    lib.loca_lowrank_truncate.argtypes = [_VP, _I64, _I64, _I64, _I64, _VP, _I64, _VP, _I64, _I64, _VP, _I64, _VP,
                                          _I64, _VP, _I64, _VP, _I64, _VP, _VP, _SZ]
    lib.loca_ridge_solve_projected.argtypes = [_VP, _I64, _I64, _I64, _I64, _VP, _VP, _I, _I64, _I64, _VP, _I64,
                                               _VP, _I64, _VP, _I64, _VP, _I64, _VP, _I64, _VP, _VP, _VP, _SZ]
    lib.loca_realization_error.argtypes = [_VP, _I64, _I64, _I64, _I64, _VP, _I64, _VP, _I64, _VP, _I, _I64, _VP,
                                           _I64, _VP, _I64, _VP, _I64, _VP, _VP, _SZ]
    lib.loca_dense_targets.argtypes = [_VP, _I64, _I64, _I64, _I64, _VP, _I64, _VP, _VP, _I64, _VP, _I64]
    lib.loca_feedback_fit.argtypes = [_VP, _I64, _I64, _I64, _I64, _VP, _VP, _I64, _D, _VP, _I, _I64, _VP, _I64,
                                      _VP, _I64, _VP, _I64, _VP, _VP, _VP, _VP, _SZ]
    lib.loca_feedback_fit_primal.argtypes = lib.loca_feedback_fit.argtypes
    lib.loca_fused_head.argtypes = [_VP, _I64, _I64, _I64, _I64, _VP, _I64, _VP, _VP, _VP, _VP, _I64, _VP, _I64, _VP,
                                    _VP, _SZ]
    lib.loca_feedback_fit_large.argtypes = [_VP, _I64, _I64, _I64, _I64, _I64, _I64, _VP, _VP, _I64, _VP, _D, _VP, _I,
                                            _I64, _VP, _I64, _VP, _I64, _VP, _I64, _VP, _VP, _VP, _VP, _SZ]
    lib.loca_top_error.argtypes = [_VP, _I64, _I64, _I64, _VP, _I, _I64, _VP, _VP, _VP, _I, _VP, _I64, _VP, _VP,
                                   _SZ]
    lib.loca_credit_from_top_error.argtypes = [_VP, _I64, _I64, _I64, _I64, _VP, _I64, _VP, _I64, _VP, _I64, _VP,
                                               _VP, _I64, _VP, _VP, _SZ]
    lib.loca_workspace_size.argtypes = [_I, _I64, _I64, _I64, _I64, _I64, _I64, _I64, _I]
    lib.loca_workspace_size.restype = _SZ
    lib.loca_status_str.argtypes = [_I]
    lib.loca_status_str.restype = ctypes.c_char_p
    lib.loca_version.restype = ctypes.c_char_p
    for name in ENTRY_POINTS:
        getattr(lib, name).restype = _I
    _lib = lib
    return lib


def status_str(s: int) -> str:
    return load().loca_status_str(s).decode()


def version() -> str:
    return load().loca_version().decode()


def workspace_size(op: int, nb: int, n: int, d: int, k: int, C: int = 0, r_a: int = 0, n_lambda: int = 0,
                   acc: int = LOCA_F32) -> int:
    return int(load().loca_workspace_size(op, nb, n, d, k, C, r_a, n_lambda, acc))


# ------------------------------------------------------------------ marshalling helpers


def _ptr(t, rows: bool = True) -> Optional[int]:
    """Device address of a tensor whose layout the C ABI describes: the last dimension
    contiguous, and with rows=True (arrays passed without a leading dimension) rows packed
    one after another.  Other layouts raise instead of being read with the wrong strides."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if t.dim() >= 1 and t.shape[-1] > 1 and t.stride(-1) != 1:
        raise ValueError(f"tensor of shape {tuple(t.shape)} and strides {t.stride()}: last dimension not contiguous")
    if rows and t.dim() >= 2 and t.shape[-2] > 1 and t.stride(-2) != t.shape[-1]:
        raise ValueError(f"tensor of shape {tuple(t.shape)} and strides {t.stride()}: rows not packed "
                         "(the C ABI takes this array without a row stride; pass a contiguous copy)")
    return t.data_ptr()


def _dtype(t) -> int:
    import torch
    return {torch.float32: LOCA_F32, torch.bfloat16: LOCA_BF16, torch.float64: LOCA_F64}[t.dtype]


def _stream(stream) -> Optional[int]:
    if stream is not None:
        return stream if isinstance(stream, int) else stream.cuda_stream
    import torch
    return torch.cuda.current_stream().cuda_stream


def _check(fn: str, st: int):
    if st != LOCA_OK:
        raise LocaError(fn, st)


def _bstride(t, nb: int) -> int:
    if t is None or nb <= 1 or isinstance(t, int):
        return 0
    return t.stride(0) if t.dim() >= 3 or (t.dim() == 2 and nb > 1 and t.shape[0] == nb) else 0


def alloc_workspace(nbytes: int, device="cuda"):
    import torch
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)


def new_mb(nb: int, device="cuda"):
    """Device array of nb loca_mb records, as a float64 tensor (nb, 4)."""
    import torch
    return torch.zeros((nb, 4), dtype=torch.float64, device=device)


def mb_view(mb):
    """(sum_q2, sum_x2, eta_bar, n) per block, as host floats."""
    import numpy as np
    h = mb.detach().cpu().numpy()
    n = h[:, 3].copy().view(np.int64)
    return {"sum_q2": h[:, 0].copy(), "sum_x2": h[:, 1].copy(), "eta_bar": h[:, 2].copy(), "n": n}


# ------------------------------------------------------------------ entry points


def loca_error_targets(logits, labels, credit_a, credit_b, y_out, mb_out, dev_info, ws, *, w=None, a_w=None,
                       e_out=None, nb=None, credit_gram=None, stream=None):
    """logits (n, C); labels (n,); credit_a (nb, C, k); credit_b (nb, k, d); y_out (nb, n, k);
    w (n,) loss weights and a_w (n,) statistic weights, float32, optional; credit_gram: B~ B~^T
    from loca_credit_gram (optional)."""
    nb = nb or credit_a.shape[0]
    n, C = logits.shape[0], logits.shape[1]
    k, d = credit_b.shape[-2], credit_b.shape[-1]
    st = load().loca_error_targets(
        _stream(stream), nb, n, C, k, d, _ptr(logits, False), _dtype(logits), logits.stride(0), _ptr(labels), _ptr(w),
        _ptr(a_w), _ptr(credit_a), _dtype(credit_a), credit_a.stride(0) if credit_a.dim() == 3 else 0, _ptr(credit_b),
        credit_b.stride(0) if credit_b.dim() == 3 else 0, _ptr(credit_gram), _ptr(y_out),
        y_out.stride(0) if y_out.dim() == 3 else 0, _ptr(e_out), _ptr(mb_out), _ptr(dev_info), _ptr(ws),
        ws.numel() * ws.element_size())
    _check("loca_error_targets", st)


def credit_gram_ld(k: int) -> int:
    return int(load().loca_credit_gram_ld(k))


def new_credit_gram(nb: int, k: int, device="cuda"):
    """Device buffer for loca_credit_gram: (nb, ld, ld) float64, ld = credit_gram_ld(k)."""
    import torch
    ld = credit_gram_ld(k)
    return torch.zeros((nb, ld, ld), dtype=torch.float64, device=device)


def loca_credit_gram(credit_b, g_out, ws, *, stream=None):
    """credit_b (nb, k, d) float32 -> g_out (nb, ld, ld) float64 = B~ B~^T per block."""
    nb, k, d = credit_b.shape
    st = load().loca_credit_gram(_stream(stream), nb, k, d, _ptr(credit_b), credit_b.stride(0), _ptr(g_out), _ptr(ws),
                                 ws.numel() * ws.element_size())
    _check("loca_credit_gram", st)


def loca_error_targets_noalloc(logits, labels, credit_a, credit_b, y_out, mb_out, dev_info, *, w=None, a_w=None,
                               e_out=None, nb=None, credit_gram=None, stream=None):
    """loca_error_targets with the library's fixed scratch array instead of a workspace."""
    nb = nb or credit_a.shape[0]
    n, C = logits.shape[0], logits.shape[1]
    k, d = credit_b.shape[-2], credit_b.shape[-1]
    st = load().loca_error_targets_noalloc(
        _stream(stream), nb, n, C, k, d, _ptr(logits, False), _dtype(logits), logits.stride(0), _ptr(labels), _ptr(w),
        _ptr(a_w), _ptr(credit_a), _dtype(credit_a), credit_a.stride(0) if credit_a.dim() == 3 else 0, _ptr(credit_b),
        credit_b.stride(0) if credit_b.dim() == 3 else 0, _ptr(credit_gram), _ptr(y_out),
        y_out.stride(0) if y_out.dim() == 3 else 0, _ptr(e_out), _ptr(mb_out), _ptr(dev_info))
    _check("loca_error_targets_noalloc", st)


def error_targets_noalloc_max_bytes() -> int:
    return int(load().loca_error_targets_noalloc_max_bytes())


def loca_accumulate_stats(x, y, eta, mb, S, K, ws, *, a_w=None, dev_info=None, overwrite=False, stream=None):
    """x (nb, n, d) bf16 or fp32 (row stride may exceed d); y (nb, n, k); S (nb, d, d); K (nb, d, k);
    a_w (n,) float32 statistic weights, the array given to loca_error_targets (optional);
    dev_info (nb,) int32 non-finite flags (optional); overwrite: S and K take this
    micro-batch's statistics instead of adding them (the first micro-batch of a step)."""
    nb, n, d = x.shape
    k = y.shape[-1]
    acc = _dtype(S)
    st = load().loca_accumulate_stats(
        _stream(stream), nb, n, d, k, _ptr(x, False), _dtype(x), x.stride(1), x.stride(0), _ptr(y), y.stride(0), _ptr(a_w),
        float(eta),
        _ptr(mb), _ptr(S), _ptr(K), acc, S.stride(0), K.stride(0), int(bool(overwrite)), _ptr(dev_info), _ptr(ws),
        ws.numel() * ws.element_size())
    _check("loca_accumulate_stats", st)


def loca_ridge_solve(S, K, lambdas: Sequence[float], m_out, dev_info, ws, *, lp=None, rp=None, credit_b=None,
                     w_dense_out=None, stream=None):
    """S (nb, d, d); K (nb, d, k); m_out (nb, n_lambda, d, r_prev + k); optional W (nb, n_lambda, d, d)."""
    nb, d, k = K.shape
    r_prev = 0 if lp is None else lp.shape[-1]
    lam = (ctypes.c_double * len(lambdas))(*[float(v) for v in lambdas])
    st = load().loca_ridge_solve(
        _stream(stream), nb, d, k, _ptr(S), _ptr(K), _dtype(S), S.stride(0), K.stride(0), _ptr(lp), _ptr(rp),
        r_prev, lp.stride(0) if lp is not None else 0, rp.stride(0) if rp is not None else 0,
        ctypes.cast(lam, ctypes.c_void_p), len(lambdas), _ptr(m_out), m_out.stride(1), _ptr(credit_b),
        credit_b.stride(0) if credit_b is not None else 0, _ptr(w_dense_out),
        w_dense_out.stride(1) if w_dense_out is not None else 0, _ptr(dev_info), _ptr(ws),
        ws.numel() * ws.element_size())
    _check("loca_ridge_solve", st)


def loca_lowrank_truncate(m, r, r_a: int, a_out, b_out, sigma_out, dev_info, ws, *, r_group=1, w_dense_out=None,
                          stream=None):
    """m (nm, d, kp); r (nr, kp, d) shared by r_group consecutive matrices; a_out (nm, r_a, d);
    b_out (nm, d, r_a); sigma_out (nm, kp)."""
    nm, d, kp = m.shape
    st = load().loca_lowrank_truncate(
        _stream(stream), nm, d, kp, r_a, _ptr(m), m.stride(0), _ptr(r), r.stride(0), r_group, _ptr(a_out),
        a_out.stride(0), _ptr(b_out), b_out.stride(0), _ptr(sigma_out), sigma_out.stride(0), _ptr(w_dense_out),
        w_dense_out.stride(0) if w_dense_out is not None else 0, _ptr(dev_info), _ptr(ws),
        ws.numel() * ws.element_size())
    _check("loca_lowrank_truncate", st)


def loca_ridge_solve_projected(S, K, credit_b, proj_a, lambdas: Sequence[float], b_out, dev_info, ws, *,
                               b_cur=None, g_out=None, stream=None):
    """S (nb, d, d); K (nb, d, k); credit_b (nb, k, d); proj_a (nb, r_a, d); b_out (nb, n_lambda, d, r_a)."""
    nb, d, k = K.shape
    r_a = proj_a.shape[-2]
    lam = (ctypes.c_double * len(lambdas))(*[float(v) for v in lambdas])
    st = load().loca_ridge_solve_projected(
        _stream(stream), nb, d, k, r_a, _ptr(S), _ptr(K), _dtype(S), S.stride(0), K.stride(0), _ptr(credit_b),
        credit_b.stride(0), _ptr(proj_a), proj_a.stride(0), _ptr(b_cur), b_cur.stride(0) if b_cur is not None else 0,
        ctypes.cast(lam, ctypes.c_void_p), len(lambdas), _ptr(b_out), b_out.stride(1), _ptr(g_out), _ptr(dev_info),
        _ptr(ws), ws.numel() * ws.element_size())
    _check("loca_ridge_solve_projected", st)


def _feedback_fit(name, e, g, beta, bt_out, sigma_out, alpha_out, dev_info, ws, wu, at_out, vk_out, stream):
    d, n_p = e.shape
    nb = g.shape[0]
    k = bt_out.shape[-2]
    vocab = wu.shape[0] if wu is not None else 0
    st = getattr(load(), name)(
        _stream(stream), nb, d, n_p, k, _ptr(e), _ptr(g), g.stride(0), float(beta), _ptr(wu),
        _dtype(wu) if wu is not None else LOCA_F32, vocab, _ptr(bt_out), bt_out.stride(0), _ptr(at_out),
        at_out.stride(0) if at_out is not None else 0, _ptr(vk_out), vk_out.stride(0) if vk_out is not None else 0,
        _ptr(sigma_out), _ptr(alpha_out), _ptr(dev_info), _ptr(ws), ws.numel() * ws.element_size())
    _check(name, st)


def loca_feedback_fit(e, g, beta: float, bt_out, sigma_out, alpha_out, dev_info, ws, *, wu=None, at_out=None,
                      vk_out=None, stream=None):
    """e (d, np) probe top errors; g (nb, d, np) exact block gradients; bt_out (nb, k, d) = B~;
    sigma_out (nb, np); alpha_out (nb,) float64; optional wu (vocab, d) and at_out (nb, vocab, k) = A~;
    optional vk_out (nb, d, k) = V_k (the factor of the paper-order head).  Dual form, np <= 64."""
    _feedback_fit("loca_feedback_fit", e, g, beta, bt_out, sigma_out, alpha_out, dev_info, ws, wu, at_out, vk_out,
                  stream)


def loca_feedback_fit_primal(e, g, beta: float, bt_out, sigma_out, alpha_out, dev_info, ws, *, wu=None,
                             at_out=None, vk_out=None, stream=None):
    """As loca_feedback_fit, through the primal form F_hat = G E^T (E E^T + beta I)^{-1}
    (np <= 128, k <= 64); the workspace is LOCA_OP_FEEDBACK_FIT_PRIMAL's."""
    _feedback_fit("loca_feedback_fit_primal", e, g, beta, bt_out, sigma_out, alpha_out, dev_info, ws, wu, at_out,
                  vk_out, stream)


def loca_feedback_fit_large(e, g, omega, q: int, beta: float, bt_out, sigma_out, alpha_out, dev_info, ws, *,
                            wu=None, at_out=None, vk_out=None, stream=None):
    """As loca_feedback_fit for any probe count (np > d included): randomised subspace iteration
    on the primal fit from the start block omega (d, l) with q rounds; sigma_out (nb, l) holds
    the Ritz values; the workspace is LOCA_OP_FEEDBACK_FIT_LARGE's (n = np, r_a = l)."""
    d, n_p = e.shape
    nb = g.shape[0]
    k = bt_out.shape[-2]
    l = omega.shape[1]
    vocab = wu.shape[0] if wu is not None else 0
    st = load().loca_feedback_fit_large(
        _stream(stream), nb, d, n_p, k, l, int(q), _ptr(e), _ptr(g), g.stride(0), _ptr(omega), float(beta),
        _ptr(wu), _dtype(wu) if wu is not None else LOCA_F32, vocab, _ptr(bt_out), bt_out.stride(0), _ptr(at_out),
        at_out.stride(0) if at_out is not None else 0, _ptr(vk_out), vk_out.stride(0) if vk_out is not None else 0,
        _ptr(sigma_out), _ptr(alpha_out), _ptr(dev_info), _ptr(ws), ws.numel() * ws.element_size())
    _check("loca_feedback_fit_large", st)


def loca_fused_head(h, wu, labels, vm, out, dev_info, ws, *, w=None, stream=None):
    """h (n, d) bf16; wu (V, d) bf16; labels (n,) int32; vm (V, c) bf16; out (n, c) float32:
    out_t = w_t (softmax(W_u h_t)^T Vm - Vm[y_t]), the logits never stored."""
    n, d = h.shape
    V = wu.shape[0]
    c = vm.shape[1]
    st = load().loca_fused_head(
        _stream(stream), n, V, d, c, _ptr(h, rows=False), h.stride(0), _ptr(wu), _ptr(labels), _ptr(w),
        _ptr(vm, rows=False), vm.stride(0), _ptr(out, rows=False), out.stride(0), _ptr(dev_info), _ptr(ws),
        ws.numel() * ws.element_size())
    _check("loca_fused_head", st)


def loca_top_error(logits, labels, wu, e_out, dev_info, ws, *, w=None, stream=None):
    """logits (n, V) f32 or bf16; labels (n,) int32; wu (V, d) bf16; e_out (n, d) float32:
    e_t = W_u^T w_t (softmax(z_t) - onehot(y_t))."""
    n, V = logits.shape
    d = wu.shape[1]
    st = load().loca_top_error(_stream(stream), n, V, d, _ptr(logits, False), _dtype(logits), logits.stride(0),
                               _ptr(labels), _ptr(w), _ptr(wu), _dtype(wu), _ptr(e_out, False), e_out.stride(0),
                               _ptr(dev_info), _ptr(ws), ws.numel() * ws.element_size())
    _check("loca_top_error", st)


def loca_credit_from_top_error(e, credit_v, credit_b, y_out, mb_out, ws, *, a_w=None, stream=None):
    """e (n, d) float32 top errors; credit_v (nb, d, k) = V_k; credit_b (nb, k, d) = B~;
    y_out (nb, n, k); a_w (n,) optional statistic weights."""
    n, d = e.shape
    nb, _, k = credit_v.shape
    st = load().loca_credit_from_top_error(_stream(stream), nb, n, d, k, _ptr(e, False), e.stride(0), _ptr(credit_v),
                                           credit_v.stride(0), _ptr(credit_b), credit_b.stride(0), _ptr(a_w),
                                           _ptr(y_out), y_out.stride(0), _ptr(mb_out), _ptr(ws),
                                           ws.numel() * ws.element_size())
    _check("loca_credit_from_top_error", st)


def loca_realization_error(m, r, K, lambdas: Sequence[float], mb_log, out, ws, *, lp=None, stream=None):
    """m (nb, n_lambda, d, kp) from loca_ridge_solve; r (nb, kp, d) = [Rp; B~]; K (nb, d, k);
    mb_log (n_mb, nb, 4) float64, the micro-batch records of the step; out (nb * n_lambda * 3,)
    float64: per (block, lambda) ||E_fit||^2, ||T||^2, ||W||^2; lp (nb, d, r_prev) or None."""
    nb, nl, d, kp = m.shape
    k = K.shape[-1]
    r_prev = 0 if lp is None else lp.shape[-1]
    assert kp == r_prev + k and mb_log.shape[1] == nb
    lam = (ctypes.c_double * len(lambdas))(*[float(v) for v in lambdas])
    st = load().loca_realization_error(
        _stream(stream), nb, d, k, r_prev, _ptr(m), m.stride(1), _ptr(r), r.stride(0), _ptr(K), _dtype(K),
        K.stride(0), _ptr(lp), lp.stride(0) if lp is not None else 0, _ptr(mb_log), mb_log.shape[0],
        ctypes.cast(lam, ctypes.c_void_p), len(lambdas), _ptr(out), _ptr(ws), ws.numel() * ws.element_size())
    _check("loca_realization_error", st)


def loca_dense_targets(y, mb, credit_b, t_out, *, stream=None):
    """y (nb, n, k); credit_b (nb, k, d); t_out (nb, n, d)."""
    nb, n, k = y.shape
    d = credit_b.shape[-1]
    st = load().loca_dense_targets(_stream(stream), nb, n, k, d, _ptr(y), y.stride(0), _ptr(mb), _ptr(credit_b),
                                   credit_b.stride(0), _ptr(t_out), t_out.stride(0))
    _check("loca_dense_targets", st)
