"""Helpers shared by the GPU parity tests: seeded inputs, the HIP path through
the C ABI, the oracle on the same inputs, and error measures."""
from __future__ import annotations

import sys
import time

import numpy as np

from paper_2608_03020_amd import inputs as gen


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def rel(a, b) -> float:
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    den = np.linalg.norm(b)
    return float(np.linalg.norm(a - b) / (den if den > 0 else 1.0))


def host_inputs(cfg, blocks, seed=0):
    """numpy inputs for the given blocks: xs[b][m], zs[m], ys[m], A[b], B[b]."""
    xs = [[gen.gen_x(cfg, b, m, seed) for m in range(cfg.n_micro)] for b in blocks]
    zs = [gen.gen_logits(cfg, m, seed) for m in range(cfg.n_micro)]
    ys = [gen.gen_labels(cfg, m, seed) for m in range(cfg.n_micro)]
    cred = [gen.gen_credit(cfg, b, seed) for b in blocks]
    return xs, zs, ys, [c[0] for c in cred], [c[1] for c in cred]


def to_dev(a, device="cuda"):
    import torch
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16).copy()).to(device).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(a)).to(device)


def padded_rows(x3, device="cuda"):
    """Device copy of x3 (nb, n, d) whose rows are padded to a 16-byte multiple (ldx >= d)."""
    nb, n, d = x3.shape
    per = 8 if x3.dtype == np.uint16 else 4
    ld = per * ((d + per - 1) // per)
    if ld == d:
        return to_dev(x3, device)
    buf = np.zeros((nb, n, ld), x3.dtype)
    buf[:, :, :d] = x3
    return to_dev(buf, device)[:, :, :d]


def run_gpu(cfg, xs, zs, ys, As, Bs, want_dense=True, proj=None, device="cuda"):
    """The HIP path over all micro-batches of len(xs) blocks; returns host arrays."""
    import torch
    from paper_2608_03020_amd import loca
    from paper_2608_03020_amd.step import BlockStep
    nb = len(xs)
    step = BlockStep(cfg, nb, device, projected=proj is not None, poison=True)
    x_all = padded_rows(np.stack([np.concatenate(xb, axis=0) for xb in xs]), device)
    z_all = to_dev(np.concatenate(zs, axis=0), device)
    y_all = to_dev(np.concatenate(ys, axis=0), device)
    A = to_dev(np.stack(As), device)
    B = to_dev(np.stack(Bs), device)
    P = to_dev(np.stack(proj), device) if proj is not None else None
    step.reset()
    Ys, mbs = [], []
    for m in range(cfg.n_micro):
        lo, hi = cfg.micro_rows(m)
        step.micro_batch(x_all[:, lo:hi], z_all[lo:hi], y_all[lo:hi], A, B)
        Ys.append(step.Y[:, :hi - lo].cpu().numpy().copy())
        mbs.append(loca.mb_view(step.mb))
    info_stats = step.info.cpu().numpy().copy()  # head error and statistics slices
    step.solve(B, P)
    nl = len(cfg.lambdas)
    # every output of the step was NaN before the calls (poisoned): none may survive
    # (S: its upper triangle, the part the statistics call maintains)
    for name, t in (("M", step.M), ("A", step.A_ad), ("B", step.B_ad), ("sigma", step.sigma),
                    ("S", torch.triu(step.S)), ("K", step.K)) + \
            ((("B_proj", step.B_proj),) if proj is not None else ()):
        assert not bool(torch.isnan(t).any()), f"{name} has unwritten (NaN) entries"
    out = {"S": step.S.cpu().numpy(), "K": step.K.cpu().numpy(), "Y": Ys, "mb": mbs,
           "M": step.M.cpu().numpy(), "sigma": step.sigma.cpu().numpy(), "A": step.A_ad.cpu().numpy(),
           "B": step.B_ad.cpu().numpy(), "info_err": info_stats, "info": step.info.cpu().numpy()}
    if proj is not None:
        out["B_proj"] = step.B_proj.cpu().numpy()
    if want_dense:
        d = cfg.d
        Wr = torch.empty((nb * nl, d, d), dtype=torch.float32, device=device)
        info = torch.zeros(nb * nl, dtype=torch.int32, device=device)
        ws = loca.alloc_workspace(loca.workspace_size(loca.LOCA_OP_LOWRANK_TRUNCATE, nb * nl, 0, d, cfg.k,
                                                      r_a=cfg.r_a), device)
        a_o = torch.full_like(step.A_ad, float("nan"))
        b_o = torch.full_like(step.B_ad, float("nan"))
        s_o = torch.full_like(step.sigma, float("nan"))
        Wr.fill_(float("nan"))
        ws.fill_(255)
        loca.loca_lowrank_truncate(step.M.view(nb * nl, d, cfg.k), B, cfg.r_a, a_o, b_o, s_o, info, ws, r_group=nl,
                                   w_dense_out=Wr)
        out["W_r"] = Wr.cpu().numpy()
        assert not np.isnan(out["W_r"]).any() and not bool(torch.isnan(a_o).any() | torch.isnan(b_o).any())
    torch.cuda.synchronize()
    return out


def run_oracle(cfg, xs_b, zs, ys, A, B, proj=None):
    """The oracle for one block (xs_b = that block's micro-batches)."""
    import oracle
    t0 = time.time()
    xf = [gen.as_f64(x, "bf16" if cfg.mode == "bf16" else "f32") for x in xs_b]
    zf = [gen.as_f64(z, cfg.logit_dtype) for z in zs]
    Af = gen.as_f64(A, cfg.a_dtype)
    res = oracle.block_step(xf, zf, ys, Af, np.asarray(B, np.float64), cfg.eta, cfg.lambdas, cfg.r_a,
                            Aproj=None if proj is None else np.asarray(proj, np.float64))
    res["seconds"] = time.time() - t0
    return res
