#!/usr/bin/env python3
"""Benchmark of the LoCA per-block adaptation step on one MI355X.

One step = one pass of the whole hot path over one batch of synthetic input
for every block of the workload: per micro-batch the head error and credit
coordinates, the streaming statistics S and K; then the ridge solves for all
ridge strengths and the rank-r_a truncation.  Inputs are resident in HBM when
the timed region starts.

Prints ONE JSON line (rank 0).  `value` = blocks * tokens / step time: the
number of (token, block) pairs taken through error -> target -> statistics ->
solve per second ("tokens/s per block").
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

BF16_PEAK_TFLOPS = 2516.6    # MI355X dense bf16 MFMA
FP64_PEAK_TFLOPS = 78.6      # MI355X dense fp64
HBM_PEAK_GBS = 8000.0

# HBM traffic of the statistics kernel (k_gram_bf16_dl) per launch, from two rocprofv3
# --pmc passes (FETCH_SIZE, then WRITE_SIZE, KiB per dispatch) of
#   bench.py --config <cfg> --steps 1 --warmup 0 --no-cpu-baseline,
# each scaled by the factor the same counter gives for a plain device copy in the same run
# (the bf16 stack of the inputs, 2 * N * d bytes read and written per block): 1.0 for both.
# Valid only for the kernel source it was taken on (digest of k_gram.hip + loca_common.h, the
# kernel file and the device helpers it includes).
TRAFFIC = {
    "c3": {"fetch_kib": 3388361.0, "write_kib": 778898.2, "fetch_scale": 1.0, "write_scale": 1.0,
           "src_digest": "8e73809de34918f3"},
    "c5": {"fetch_kib": 15697122.3, "write_kib": 2700420.1, "fetch_scale": 1.0, "write_scale": 1.0,
           "src_digest": "8e73809de34918f3"},
}


def stats_src_digest():
    import hashlib
    h = hashlib.sha256()
    for f in ("k_gram.hip", "loca_common.h"):
        with open(os.path.join(ROOT, "paper_2608_03020_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def traffic_bytes(cfg_name):
    t = TRAFFIC.get(cfg_name)
    if t is None or t["src_digest"] != stats_src_digest():
        return None
    return 1024.0 * (t["fetch_kib"] * t["fetch_scale"] + t["write_kib"] * t["write_scale"])


WORKLOADS = {
    "c1": "Single block, Qwen2.5-0.5B width: d=896, N=512, C=2, k=8, r_a=8, lambda=1e-2, fp32 mode",
    "c2": "Qwen2.5-1.5B-shaped: 28 blocks, d=1536, N=8192 (4 x 2048), C=4, k=16, r_a=16, lambda=1e-2, bf16 X",
    "c3": "Qwen2.5-7B-shaped: 28 blocks, d=3584, N=32768 (4 x 8192), C=5, k=32, r_a=16, "
          "lambda in {1e-3,1e-2,1e-1}, bf16 X, fp32 accumulation",
    "c4": "Full-vocabulary error: 1 block, d=2048, N=4096, V=151936 (bf16 logits), k=64, r_a=32, bf16 X",
    "c5": "Qwen2.5-14B-shaped: 48 blocks, d=5120, N=65536 (8 x 8192), C=5, k=64, r_a=32, lambda=1e-2, bf16 X",
}


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=10)
    p.add_argument("--warmup", type=int, default=2)
    p.add_argument("--config", default="c5", choices=sorted(WORKLOADS),
                   help="headline workload (default c5, the largest configuration)")
    p.add_argument("--secondary", default="c3", type=lambda v: [x for x in v.split(",") if x],
                   help="comma-separated workloads timed after the headline and reported under "
                        "\"secondary\" (default c3, the first at d >= 3584; '' for none)")
    p.add_argument("--blocks", type=int, default=0, help="override the block count (profiling runs)")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-tokens", type=int, default=0, help="tokens in the CPU-baseline sample")
    p.add_argument("--next", action="store_true",
                   help="also time the widened rows (weighted statistics, outer step with a current adapter, "
                        "Stage I calibration on the same workload; the paper-order head on a full-vocabulary "
                        "workload with 24 blocks)")
    return p.parse_args()


def make_inputs(cfg, nb, device="cuda"):
    import numpy as np
    import torch
    from paper_2608_03020_amd import inputs as gen
    xs = []
    A = []
    B = []
    for b in range(nb):
        x, a, bb = gen.torch_gen_block_inputs(cfg, b, seed=0, device=device)
        xs.append(x)
        A.append(a)
        B.append(bb)
    x_all = torch.stack(xs)
    del xs
    z, y = gen.torch_gen_head(cfg, seed=0, device=device)
    return x_all, z, y, torch.stack(A), torch.stack(B)


def run_step(step, cfg, nb, x_all, z, y, A, B, stream, record=None, a_all=None, lp=None, rp=None,
             solve_record=None, error_record=None, proj=None):
    """One step of the whole path over every block: per micro-batch the head error
    and credit coordinates (from the event error_record[m] when given), then the
    statistics (bracketed by the events of `record[m]` when given); then the ridge
    solves, the truncation and, with the projections `proj` (nb, r_a, d), the
    paper-literal projected solve, which needs only the statistics and runs on a stream
    of its own beside the ridge solves (bracketed by `solve_record`: start, between the
    solves and the truncation and after the truncation when it has four events, end,
    after the step's stream has waited for the projected solve).  Optional: statistic
    weights a_all (n,), a current adapter lp (nb, d, r_prev), rp (nb, r_prev, d)."""
    from paper_2608_03020_amd import loca
    step.reset()
    for m in range(cfg.n_micro):
        lo, hi = cfg.micro_rows(m)
        xm = x_all[:, lo:hi]
        yv = step.Y[:, :hi - lo]
        aw = None if a_all is None else a_all[lo:hi]
        if error_record is not None:
            error_record[m].record(stream)
        if m == 0:  # B~ B~^T once per step, shared by the micro-batches
            loca.loca_credit_gram(B, step.G, step.ws)
        loca.loca_error_targets(z[lo:hi], y[lo:hi], A, B, yv, step.mb, step.info_err[m:m + 1], step.ws, a_w=aw,
                                nb=nb, credit_gram=step.G)
        if record is not None:
            record[m][0].record(stream)
        loca.loca_accumulate_stats(xm, yv, cfg.eta, step.mb, step.S, step.K, step.ws, a_w=aw,
                                   dev_info=step.info_stats[m], overwrite=m == 0)
        if record is not None:
            record[m][1].record(stream)
    if solve_record is not None:
        solve_record[0].record(stream)
    marks = solve_record if solve_record is not None and len(solve_record) == 4 else None
    step.solve(B, proj_a=proj, lp=lp, rp=rp, mid_event=marks[1] if marks else None,
               trunc_event=marks[2] if marks else None)
    if solve_record is not None:
        solve_record[-1].record(stream)


def stats_flops(cfg, nb):
    """Algorithmic flops of every statistics call of one step (d(d+1) + 2dk per token and block)."""
    rows = [cfg.micro_rows(m)[1] - cfg.micro_rows(m)[0] for m in range(cfg.n_micro)]
    return [nb * (r * cfg.d * (cfg.d + 1) + 2 * r * cfg.d * cfg.k) for r in rows]


def solve_flops(cfg, nb, r_prev):
    """Algorithmic flops of the ridge solves of one step: per block and lambda the Cholesky
    d^3/3, the right-hand sides S Lp (2 d^2 r_prev) and the two triangular solves (2 d^2 kp)."""
    d, kp = cfg.d, r_prev + cfg.k
    return nb * len(cfg.lambdas) * (d ** 3 / 3.0 + 2.0 * d * d * r_prev + 2.0 * d * d * kp)


def time_steps(fn, steps, warmup):
    import torch
    for _ in range(warmup):
        fn(0)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(steps):
        fn(s)
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) * 1e3 / steps


def next_rows(args, cfg, nb, x_all, z, y, A, B, step, stream):
    """The widened rows on the same workload and inputs: statistic weights on every
    micro-batch (Section S7's weighted form), the outer step past the first with a
    rank-r_a current adapter (Theorem S6.1), and the Stage I calibration of all blocks
    from 64 probe pairs (Section S5).  Each with its time and the roofline of the call
    that dominates it."""
    import numpy as np
    import torch
    from paper_2608_03020_amd import inputs as gen
    from paper_2608_03020_amd import loca
    from paper_2608_03020_amd.step import BlockStep
    out = {}
    steps = max(1, min(args.steps, 5))
    n_mb = cfg.n_micro
    peak = FP64_PEAK_TFLOPS if cfg.mode == "fp32" else BF16_PEAK_TFLOPS

    # weighted statistics: same workload, a_t uniform on [0, 2) with 20% zeros
    a_all = gen.torch_gen_stat_weights(cfg)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps * n_mb)]
    ms = time_steps(lambda s: run_step(step, cfg, nb, x_all, z, y, A, B, stream,
                                       ev[s * n_mb:(s + 1) * n_mb] if s < steps else None, a_all=a_all),
                    steps, 1)
    t_avg = sum(a.elapsed_time(b) for a, b in ev) / len(ev)
    f_avg = sum(stats_flops(cfg, nb)) / n_mb
    ach = f_avg / (t_avg * 1e-3) / 1e12
    out["weighted_statistics"] = {
        "ms_per_step": ms, "value": nb * cfg.n / (ms * 1e-3), "unit": "tokens/s per block",
        "weights": "a_t uniform on [0, 2), 20% zero, every micro-batch",
        "roofline": {"bound": "mfma", "achieved": ach, "peak": peak, "unit": "TFLOP/s", "frac": ach / peak,
                     "traffic": None, "kernel": "loca_accumulate_stats with statistic weights (all blocks, one micro-batch)",
                     "algorithmic_flops_per_launch": f_avg, "avg_launch_ms": t_avg}}
    print(f"[bench] next: weighted statistics {ms:.2f} ms/step", file=sys.stderr, flush=True)
    del a_all

    # outer step with a current adapter W_prev = Lp Rp of rank r_a
    r_prev = cfg.r_a
    if r_prev + cfg.k <= 128:
        lp, rp = gen.torch_gen_current_adapter(cfg, nb, r_prev)
        step2 = BlockStep(cfg, nb, torch.device("cuda:0"), r_prev=r_prev)
        sev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
        ms = time_steps(lambda s: run_step(step2, cfg, nb, x_all, z, y, A, B, stream, lp=lp, rp=rp,
                                           solve_record=sev[s] if s < steps else None), steps, 1)
        t_solve = sum(a.elapsed_time(b) for a, b in sev) / len(sev)
        fl = solve_flops(cfg, nb, r_prev)
        ach = fl / (t_solve * 1e-3) / 1e12
        pk = FP64_PEAK_TFLOPS if cfg.mode == "fp32" else 157.3
        out["outer_step_current_adapter"] = {
            "ms_per_step": ms, "value": nb * cfg.n / (ms * 1e-3), "unit": "tokens/s per block", "r_prev": r_prev,
            "roofline": {"bound": "mfma", "achieved": ach, "peak": pk, "unit": "TFLOP/s", "frac": ach / pk,
                         "traffic": None,
                         "kernel": "ridge solves (all blocks and lambdas, right-hand sides [S Lp | K]) and truncation",
                         "algorithmic_flops_per_launch": fl, "avg_launch_ms": t_solve}}
        print(f"[bench] next: outer step {ms:.2f} ms/step (solve + truncation {t_solve:.2f} ms)", file=sys.stderr,
              flush=True)
        del step2, lp, rp
        torch.cuda.empty_cache()

    # Stage I calibration of every block from 64 probe pairs
    n_p, k, V = 64, cfg.k, cfg.C
    E, G = gen.torch_gen_probe_pairs(cfg, n_p, nb)
    g = torch.Generator(device="cuda")
    g.manual_seed(7)
    Wu = torch.randn((V, cfg.d), generator=g, device="cuda", dtype=torch.float32) / np.sqrt(cfg.d)
    bt = torch.empty((nb, k, cfg.d), dtype=torch.float32, device="cuda")
    at = torch.empty((nb, V, k), dtype=torch.float32, device="cuda")
    sig = torch.empty((nb, n_p), dtype=torch.float32, device="cuda")
    alpha = torch.empty(nb, dtype=torch.float64, device="cuda")
    info = torch.empty(nb, dtype=torch.int32, device="cuda")
    ws = loca.alloc_workspace(loca.workspace_size(loca.LOCA_OP_FEEDBACK_FIT, nb, n_p, cfg.d, k), "cuda")
    reps = 20
    cev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]

    def calib(s):
        if s < reps:
            cev[s][0].record(stream)
        loca.loca_feedback_fit(E, G, 0.05, bt, sig, alpha, info, ws, wu=Wu, at_out=at)
        if s < reps:
            cev[s][1].record(stream)
    time_steps(calib, reps, 2)
    t_cal = sum(a.elapsed_time(b) for a, b in cev) / reps
    nbytes = 4.0 * (cfg.d * n_p + nb * cfg.d * n_p + nb * k * cfg.d + nb * V * k + V * cfg.d)
    gbs = nbytes / (t_cal * 1e-3) / 1e9
    cal = {"ms_per_call": t_cal, "unit": "ms per calibration of all blocks", "higher_is_better": False,
           "config": {"blocks": nb, "d": cfg.d, "probes": n_p, "credit_rank": k, "head_rows": V, "beta": 0.05},
           "alpha_mean": float(alpha.mean().item()),
           "roofline": {"bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": gbs / HBM_PEAK_GBS,
                        "traffic": None, "kernel": "loca_feedback_fit (all blocks)",
                        "algorithmic_bytes_per_launch": nbytes, "avg_launch_ms": t_cal}}
    print(f"[bench] next: calibration {t_cal:.3f} ms", file=sys.stderr, flush=True)
    if not args.no_cpu_baseline:
        # the oracle forms the d x d map and takes its full SVD (O(d^3)): timed on the first
        # d_s rows and columns of block 0's probes and scaled by (d / d_s)^3 and the block count
        import oracle
        d_s = min(cfg.d, 1024)
        print(f"[bench] next: cpu baseline of the calibration (oracle, width {d_s})", file=sys.stderr, flush=True)
        E_h = E[:d_s].double().cpu().numpy()
        G_h = G[0, :d_s].double().cpu().numpy()
        W_h = Wu[:, :d_s].double().cpu().numpy()
        t0 = time.perf_counter()
        F = oracle.feedback_fit(E_h, G_h, 0.05)
        F_k, _, _, _ = oracle.feedback_factors(F, k, W_h)
        oracle.alignment(F_k, E_h, G_h)
        t_blk = time.perf_counter() - t0
        scale = (cfg.d / d_s) ** 3 * nb
        cal["cpu_baseline"] = {"value": t_blk * scale * 1e3, "unit": "ms per calibration of all blocks",
                               "cores": int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1)),
                               "kind": "oracle",
                               "sample": f"block 0 at width {d_s} with {n_p} probes ({t_blk:.2f} s), scaled by "
                                         f"(d/{d_s})^3 x {nb} blocks"}
    out["feedback_fit"] = cal
    del E, G, bt, at, ws
    torch.cuda.empty_cache()

    # Stage I calibration from 2d probe positions (np > d: a full-rank d x d fitted map),
    # randomised subspace iteration of width l = min(2k, 128) with q = 3 rounds
    n_p, l, q = 2 * cfg.d, min(2 * k, 128), 3
    E, G = gen.torch_gen_probe_pairs(cfg, n_p, nb)
    omega = torch.randn((cfg.d, l), generator=g, device="cuda", dtype=torch.float32)
    bt = torch.empty((nb, k, cfg.d), dtype=torch.float32, device="cuda")
    at = torch.empty((nb, V, k), dtype=torch.float32, device="cuda")
    sig = torch.empty((nb, l), dtype=torch.float32, device="cuda")
    ws = loca.alloc_workspace(loca.workspace_size(loca.LOCA_OP_FEEDBACK_FIT_LARGE, nb, n_p, cfg.d, k, r_a=l), "cuda")
    reps_l = 2
    lev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps_l)]

    def calib_large(s):
        if s < reps_l:
            lev[s][0].record(stream)
        loca.loca_feedback_fit_large(E, G, omega, q, 0.05, bt, sig, alpha, info, ws, wu=Wu, at_out=at)
        if s < reps_l:
            lev[s][1].record(stream)
    time_steps(calib_large, reps_l, 1)
    t_l = sum(a.elapsed_time(b) for a, b in lev) / reps_l
    d_ = cfg.d
    # algorithmic float64 flops: E E^T, one factorisation, the triangular solves (the np
    # columns of E when R is formed, or l columns per block and product when it is applied,
    # whichever takes fewer solves of at most 128 columns), the 2q + 2 products with F_hat or
    # F_hat^T (two skinny products each), 2q + 1 two-pass Cholesky QRs (Gram and basis
    # update), and the alignment products
    applied = 2 * (q + 1) * nb < -(-n_p // 128)
    solve_cols = (2 * q + 2) * nb * l if applied else n_p
    fl = (2.0 * d_ * d_ * n_p + d_ ** 3 / 3.0 + 2.0 * d_ * d_ * solve_cols
          + nb * ((2 * q + 2) * 4.0 * d_ * n_p * l + (2 * q + 1) * 2 * 4.0 * d_ * l * l + 4.0 * k * d_ * n_p))
    tfs = fl / (t_l * 1e-3) / 1e12
    out["feedback_fit_large"] = {
        "ms_per_call": t_l, "unit": "ms per calibration of all blocks", "higher_is_better": False,
        "config": {"blocks": nb, "d": d_, "probes": n_p, "credit_rank": k, "basis": l, "rounds": q,
                   "head_rows": V, "beta": 0.05, "R": "applied" if applied else "formed"},
        "info_ok": bool((info == 0).all().item()), "alpha_mean": float(alpha.mean().item()),
        "roofline": {"bound": "alu", "achieved": tfs, "peak": FP64_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": tfs / FP64_PEAK_TFLOPS, "traffic": None, "kernel": "loca_feedback_fit_large (all blocks)",
                     "algorithmic_flops_per_call": fl, "avg_launch_ms": t_l}}
    print(f"[bench] next: calibration with {n_p} probes {t_l:.1f} ms", file=sys.stderr, flush=True)
    del E, G, Wu, bt, at, ws, omega
    torch.cuda.empty_cache()
    out["paper_order_head"] = paper_order_head(stream)
    out["fused_head"] = fused_head_rows(stream)
    return out


def paper_order_head(stream, L=24, d=896, n=4096, V=151936, k=64, reps=5):
    """The head in the paper's order on a full-vocabulary workload with many blocks
    (Qwen2.5-0.5B shape: 24 blocks of width 896, 151936-token vocabulary, k = 64, so
    L k > d): the top error e = W_u^T E once plus V_k^T e per block, against the folded
    order (A~ = W_u V_k per block in the error kernel) on the same logits."""
    import numpy as np
    import torch
    from paper_2608_03020_amd import loca
    g = torch.Generator(device="cuda")
    g.manual_seed(11)
    z = (torch.randn((n, V), generator=g, device="cuda") * 2.0).to(torch.bfloat16)
    y = torch.randint(0, V, (n,), generator=g, device="cuda", dtype=torch.int32)
    Wu = (torch.randn((V, d), generator=g, device="cuda") / np.sqrt(d)).to(torch.bfloat16)
    Vk = torch.randn((L, d, k), generator=g, device="cuda") / np.sqrt(d)
    Bt = torch.randn((L, k, d), generator=g, device="cuda") / np.sqrt(k)
    At = torch.stack([(Wu.float() @ Vk[b]).to(torch.bfloat16) for b in range(L)])
    e = torch.empty((n, d), dtype=torch.float32, device="cuda")
    Y = torch.empty((L, n, k), dtype=torch.float32, device="cuda")
    mb = loca.new_mb(L, "cuda")
    info = torch.zeros(1, dtype=torch.int32, device="cuda")
    ws = loca.alloc_workspace(max(loca.workspace_size(loca.LOCA_OP_TOP_ERROR, 1, n, d, 1, V),
                                  loca.workspace_size(loca.LOCA_OP_CREDIT_FROM_TOP_ERROR, L, n, d, k),
                                  loca.workspace_size(loca.LOCA_OP_ERROR_TARGETS, L, n, d, k, V)), "cuda")
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(reps)]

    def paper(s):
        if s < reps:
            ev[s][0].record(stream)
        loca.loca_top_error(z, y, Wu, e, info, ws)
        if s < reps:
            ev[s][1].record(stream)
        loca.loca_credit_from_top_error(e, Vk, Bt, Y, mb, ws)
        if s < reps:
            ev[s][2].record(stream)

    def folded(s):
        loca.loca_error_targets(z, y, At, Bt, Y, mb, info, ws, nb=L)
        if s < reps:
            ev[s][3].record(stream)
    ms_paper = time_steps(paper, reps, 1)
    ms_folded = time_steps(folded, reps, 1)
    t_top = sum(a[0].elapsed_time(a[1]) for a in ev) / reps
    t_cred = sum(a[1].elapsed_time(a[2]) for a in ev) / reps
    fl = 2.0 * n * V * d
    ach = fl / (t_top * 1e-3) / 1e12
    print(f"[bench] next: paper-order head {ms_paper:.2f} ms (top error {t_top:.2f} ms), folded {ms_folded:.2f} ms",
          file=sys.stderr, flush=True)
    return {"config": {"blocks": L, "d": d, "tokens": n, "vocab": V, "credit_rank": k, "logits": "bf16",
                       "head": "bf16"},
            "ms_paper_order": ms_paper, "ms_folded_order": ms_folded, "ms_top_error": t_top,
            "ms_credit_all_blocks": t_cred, "speedup_vs_folded": ms_folded / ms_paper,
            "roofline": {"bound": "mfma", "achieved": ach, "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                         "frac": ach / BF16_PEAK_TFLOPS, "traffic": None,
                         "kernel": "loca_top_error (softmax statistics, the split-K product e = W_u^T E, reduction)",
                         "algorithmic_flops_per_launch": fl, "avg_launch_ms": t_top}}


def fused_head_rows(stream, n=4096, V=151936, reps=5):
    """The fused LM head from hidden states (logits never stored) on the two full-vocabulary
    shapes: the folded order of one Qwen2.5-3B-width block (d = 2048, Vm = A~, k = 64) and
    the paper's order at the 0.5B width (d = 896, Vm = W_u: the top error, then V_k^T e for
    24 blocks)."""
    import numpy as np
    import torch
    from paper_2608_03020_amd import loca
    rows = {}
    for name, d, k, L in (("folded_d2048_k64", 2048, 64, 1), ("paper_order_d896_L24_k64", 896, 64, 24)):
        g = torch.Generator(device="cuda")
        g.manual_seed(12)
        h = (torch.randn((n, d), generator=g, device="cuda") * 2.0).to(torch.bfloat16)
        y = torch.randint(0, V, (n,), generator=g, device="cuda", dtype=torch.int32)
        Wu = (torch.randn((V, d), generator=g, device="cuda") / np.sqrt(d)).to(torch.bfloat16)
        paper = name.startswith("paper")
        if paper:
            Vm = Wu
            Vk = torch.randn((L, d, k), generator=g, device="cuda") / np.sqrt(d)
            Bt = torch.randn((L, k, d), generator=g, device="cuda") / np.sqrt(k)
            Y = torch.empty((L, n, k), dtype=torch.float32, device="cuda")
            mb = loca.new_mb(L, "cuda")
        else:
            Vm = (Wu.float() @ (torch.randn((d, k), generator=g, device="cuda") / np.sqrt(d))).to(torch.bfloat16)
        c = Vm.shape[1]
        out = torch.empty((n, c), dtype=torch.float32, device="cuda")
        info = torch.zeros(1, dtype=torch.int32, device="cuda")
        nbytes = loca.workspace_size(loca.LOCA_OP_FUSED_HEAD, 1, n, d, c, V)
        if paper:
            nbytes = max(nbytes, loca.workspace_size(loca.LOCA_OP_CREDIT_FROM_TOP_ERROR, L, n, d, k))
        ws = loca.alloc_workspace(nbytes, "cuda")
        ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(reps)]

        def call(s):
            if s < reps:
                ev[s][0].record(stream)
            loca.loca_fused_head(h, Wu, y, Vm, out, info, ws)
            if s < reps:
                ev[s][1].record(stream)
            if paper:
                loca.loca_credit_from_top_error(out, Vk, Bt, Y, mb, ws)
        ms = time_steps(call, reps, 1)
        t_f = sum(a[0].elapsed_time(a[1]) for a in ev) / reps
        fl = 2.0 * n * V * (d + c)
        ach = fl / (t_f * 1e-3) / 1e12
        rows[name] = {"config": {"tokens": n, "vocab": V, "d": d, "columns": c, "blocks": L, "credit_rank": k},
                      "ms_per_call": ms, "ms_fused_head": t_f, "info_ok": int(info.item()) == 0,
                      "roofline": {"bound": "mfma", "achieved": ach, "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                                   "frac": ach / BF16_PEAK_TFLOPS, "traffic": None,
                                   "kernel": "loca_fused_head (logits on the matrix cores, online softmax, E Vm)",
                                   "algorithmic_flops_per_launch": fl, "avg_launch_ms": t_f}}
        print(f"[bench] next: fused head {name}: {t_f:.2f} ms ({ach / BF16_PEAK_TFLOPS:.3f} of bf16 peak)",
              file=sys.stderr, flush=True)
        del h, Wu, Vm, out, ws
        torch.cuda.empty_cache()
    return rows


def cpu_baseline(cfg, n_sample):
    """The oracle as it stands, on a bounded sample of block 0 of the workload:
    the per-token stages (head error, feedback, target, S, dense Z, K, the projected
    statistics) on `n_sample` tokens of one micro-batch, scaled to the block's N
    tokens, plus the per-block stages (ridge solve of every lambda with the factored
    right-hand side K, Eckart-Young truncation, projected solve) at full width."""
    import numpy as np
    import oracle
    from paper_2608_03020_amd import inputs as gen
    threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    sub = gen.custom_config("sample", blocks=1, d=cfg.d, n=n_sample, C=cfg.C, k=cfg.k, r_a=cfg.r_a,
                            lambdas=cfg.lambdas, mode=cfg.mode, x_dist=cfg.x_dist, n_outlier=cfg.n_outlier,
                            outlier_scale=cfg.outlier_scale, logit_std=cfg.logit_std, logit_dtype=cfg.logit_dtype,
                            a_dtype=cfg.a_dtype, eta=cfg.eta)
    X = gen.as_f64(gen.gen_x(sub, 0, 0), "bf16" if cfg.mode == "bf16" else "f32")
    z = gen.as_f64(gen.gen_logits(sub, 0), cfg.logit_dtype)
    y = gen.gen_labels(sub, 0)
    A, Bm = gen.gen_credit(sub, 0)
    A = gen.as_f64(A, cfg.a_dtype)
    Bm = np.asarray(Bm, np.float64)
    Ap = np.asarray(gen.gen_adapter_projection(sub, 0), np.float64)
    t0 = time.perf_counter()
    E = oracle.head_error(z, y)
    Y, Q = oracle.credit(E, A, Bm)
    T, info = oracle.scaled_target(X, Q, cfg.eta)
    S = oracle.gram_acc(X)
    Z = oracle.cross_acc(X, T)
    K = oracle.cross_acc(X, -info["eta_bar"] * Y)
    G, Cst = oracle.projected_acc(X, T, Ap)
    t_tok = time.perf_counter() - t0
    # per-block stages on a well-posed full-width system (the sample's S has rank n_sample < d)
    S_full = S + np.eye(cfg.d) * float(np.trace(S) / cfg.d)
    t1 = time.perf_counter()
    Ms = [oracle.ridge_solve(S_full, K, lam)[0] for lam in cfg.lambdas]
    for M in Ms:
        oracle.truncate_factored(M, Bm, cfg.r_a, want_dense=False)
    G_full = G + np.eye(cfg.r_a) * float(np.trace(G) / cfg.r_a)
    for lam in cfg.lambdas:
        oracle.projected_solve(G_full, Cst, lam)
    t_blk = time.perf_counter() - t1
    t_block = t_tok * (cfg.n / n_sample) + t_blk
    return {"value": cfg.n / t_block, "unit": "tokens/s per block", "cores": threads, "kind": "oracle",
            "sample": (f"block 0 of {cfg.name}: per-token stages on {n_sample} of {cfg.n} tokens "
                       f"({t_tok:.2f} s, scaled x{cfg.n / n_sample:.0f}); ridge solves for {len(cfg.lambdas)} "
                       f"lambda(s) with the factored right-hand side, truncation and projected solve at d={cfg.d} "
                       f"({t_blk:.2f} s)"),
            "seconds_per_block": t_block, "_unused": float(Z[0, 0])}


def measure(args, name, nb_override=0, keep=False):
    """Time args.steps steps of the whole path on workload `name` (after args.warmup
    untimed ones): inputs resident in HBM, HIP events around every statistics call and
    the step's phases.  Returns the JSON fields of the line; with keep=True also the
    device state (for the widened rows)."""
    import numpy as np
    import torch
    from paper_2608_03020_amd import inputs as gen
    from paper_2608_03020_amd.inputs import CONFIGS
    from paper_2608_03020_amd.step import BlockStep

    cfg = CONFIGS[name]
    nb = nb_override or cfg.blocks
    dev = torch.device("cuda:0")
    print(f"[bench] {name}: generating inputs for {nb} blocks", file=sys.stderr, flush=True)
    x_all, z, y, A, B = make_inputs(cfg, nb)
    proj = gen.torch_gen_adapter_projection(cfg, nb)
    step = BlockStep(cfg, nb, dev, projected=True)
    stream = torch.cuda.current_stream()
    torch.cuda.synchronize()

    # events around every statistics call of the timed region (the dominant kernel)
    n_mb = cfg.n_micro
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps * n_mb)]
    ev_err = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps * n_mb)]
    ev_sol = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]

    def one_step(record=None, s=None):
        run_step(step, cfg, nb, x_all, z, y, A, B, stream, record,
                 solve_record=ev_sol[s] if s is not None else None,
                 error_record=ev_err[s * n_mb:(s + 1) * n_mb] if s is not None else None, proj=proj)

    for _ in range(args.warmup):
        one_step()
    torch.cuda.synchronize()
    print(f"[bench] {name}: warmup done; timing {args.steps} steps", file=sys.stderr, flush=True)
    t0 = time.perf_counter()
    for s in range(args.steps):
        one_step(ev[s * n_mb:(s + 1) * n_mb], s)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    ms_step = dt * 1e3 / args.steps
    info = step.info.cpu().numpy()
    if np.any(info != 0):
        print(f"[bench] warning: dev_info {info}", file=sys.stderr)

    stats_ms = [a.elapsed_time(b) for a, b in ev]
    flops = stats_flops(cfg, nb) * args.steps
    t_avg = sum(stats_ms) / len(stats_ms)
    f_avg = sum(flops) / len(flops)
    achieved = f_avg / (t_avg * 1e-3) / 1e12
    peak = FP64_PEAK_TFLOPS if cfg.mode == "fp32" else BF16_PEAK_TFLOPS
    K = args.steps
    breakdown = {
        "unit": "ms per step (HIP events on the launch stream)",
        "head_error_and_coordinates": sum(ev_err[i].elapsed_time(ev[i][0]) for i in range(K * n_mb)) / K,
        "statistics": sum(stats_ms) / K,
        "ridge_solves": sum(e[0].elapsed_time(e[1]) for e in ev_sol) / K,
        "truncation": sum(e[1].elapsed_time(e[2]) for e in ev_sol) / K,
        "wait_for_projected_solve": sum(e[2].elapsed_time(e[3]) for e in ev_sol) / K,
    }
    out = {
        "value": nb * cfg.n / (ms_step * 1e-3),
        "ms_per_step": ms_step,
        "dtype": "f64" if cfg.mode == "fp32" else "bf16",
        "config": {"workload": f"{name}: {WORKLOADS[name]}", "blocks": nb, "d": cfg.d,
                   "tokens": cfg.n, "micro_batch": cfg.micro, "classes": cfg.C, "credit_rank": cfg.k,
                   "adapter_rank": cfg.r_a, "lambdas": list(cfg.lambdas)},
        "roofline": {"bound": "mfma", "achieved": achieved, "peak": peak, "unit": "TFLOP/s",
                     "frac": achieved / peak, "traffic": traffic_bytes(name),
                     "kernel": "loca_accumulate_stats (Gram S += X^T X and cross X^T Y of all blocks, one micro-batch)",
                     "algorithmic_flops_per_launch": f_avg, "avg_launch_ms": t_avg},
        "breakdown": breakdown,
    }
    if keep:
        return out, (cfg, nb, x_all, z, y, A, B, step, stream)
    del x_all, z, y, A, B, proj, step
    torch.cuda.empty_cache()
    return out, None


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py: the library runs on one GPU; --gpus {args.gpus} is not supported "
              "(sharding the blocks across GPUs is described, not implemented).", file=sys.stderr)
        sys.exit(2)
    import torch
    torch.cuda.init()

    head, state = measure(args, args.config, args.blocks, keep=args.next)
    out = {
        "metric": "tokens/sec per block (error->target->Gram+solve); % MFMA peak on X^T X",
        "value": head["value"],
        "unit": "tokens/s per block",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": head["dtype"],
        "data": "synthetic (seeded; device-generated inputs with the workload's distributions)",
        "config": head["config"],
        "roofline": head["roofline"],
        "breakdown": head["breakdown"],
    }
    if args.next:
        cfg, nb, x_all, z, y, A, B, step, stream = state
        out["next"] = next_rows(args, cfg, nb, x_all, z, y, A, B, step, stream)
        del state, x_all, z, y, A, B, step
        torch.cuda.empty_cache()
    for name in args.secondary:
        if name != args.config:
            row, _ = measure(args, name)
            out.setdefault("secondary", {})[name] = row
    if not args.no_cpu_baseline:
        from paper_2608_03020_amd.inputs import CONFIGS
        cfg = CONFIGS[args.config]
        n_s = args.cpu_tokens or (512 if cfg.d >= 3000 else 1024)
        print(f"[bench] cpu baseline: oracle on {n_s} tokens", file=sys.stderr, flush=True)
        cb = cpu_baseline(cfg, min(n_s, cfg.n))
        cb.pop("_unused", None)
        out["cpu_baseline"] = cb
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
