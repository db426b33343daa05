"""One pass of the per-block adaptation step over all blocks of a workload.

Owns the device buffers (torch) and issues the C-ABI calls in the order of
the outer iteration (Section S13, steps 2-5): for every micro-batch the head
error and credit coordinates, then the streaming statistics; then the ridge
solves for every lambda; then the rank-r_a truncation.  Orchestration only:
all arithmetic runs in libloca's kernels.
"""
from __future__ import annotations

from typing import List, Optional

from . import loca
from .inputs import LocaConfig


class BlockStep:
    """Buffers and calls for `nb` blocks of a config, micro-batch by micro-batch.

    x_blocks: device tensor (nb, n, d) with all micro-batches of every block
    (bf16 or fp32); logits (n, C); labels (n,); credit_a (nb, C, k);
    credit_b (nb, k, d).
    """

    def __init__(self, cfg: LocaConfig, nb: int, device="cuda", projected: bool = False, n_total: Optional[int] = None,
                 r_prev: int = 0, poison: bool = False):
        import torch
        self.cfg, self.nb, self.device = cfg, nb, device
        d, k, r_a = cfg.d, cfg.k, cfg.r_a
        nl = len(cfg.lambdas)
        acc_t = torch.float64 if cfg.mode == "fp32" else torch.float32
        self.acc = loca.LOCA_F64 if cfg.mode == "fp32" else loca.LOCA_F32
        n_mb = cfg.micro
        self.S = torch.zeros((nb, d, d), dtype=acc_t, device=device)
        self.K = torch.zeros((nb, d, k), dtype=acc_t, device=device)
        self.Y = torch.empty((nb, n_mb, k), dtype=torch.float32, device=device)
        self.mb = loca.new_mb(nb, device)
        self.G = loca.new_credit_gram(nb, k, device)  # B~ B~^T, formed once per step
        self.mb_log: List = []
        # one dev_info slice per call, so that no call's codes overwrite another's: the head
        # error of every micro-batch, the statistics of every (micro-batch, block), the solve,
        # the truncation and the projected solve of every (block, lambda)
        i32 = dict(dtype=torch.int32, device=device)
        self.info_err = torch.zeros(cfg.n_micro, **i32)
        self.info_stats = torch.zeros((cfg.n_micro, nb), **i32)
        self.info_solve = torch.zeros(nb * nl, **i32)
        self.info_trunc = torch.zeros(nb * nl, **i32)
        self.info_proj = torch.zeros(nb * nl, **i32)
        self._m = 0
        self._gram = False
        self.r_prev = r_prev
        kp = r_prev + k  # right-hand sides of the solve: [S Lp | K]
        self.M = torch.empty((nb, nl, d, kp), dtype=torch.float32, device=device)
        self.A_ad = torch.empty((nb * nl, r_a, d), dtype=torch.float32, device=device)
        self.B_ad = torch.empty((nb * nl, d, r_a), dtype=torch.float32, device=device)
        self.sigma = torch.empty((nb * nl, kp), dtype=torch.float32, device=device)
        self.projected = projected
        if projected:
            self.B_proj = torch.empty((nb, nl, d, r_a), dtype=torch.float32, device=device)
            # the projected solve reads only the statistics: it runs on a stream of its own
            # (default priority) beside the ridge solves, with a workspace of its own
            self.ws_proj = loca.alloc_workspace(
                loca.workspace_size(loca.LOCA_OP_RIDGE_SOLVE_PROJECTED, nb, n_mb, d, k, cfg.C, r_a, nl, self.acc),
                device)
            self.side = torch.cuda.Stream(device=device)
        ws = max(
            loca.workspace_size(loca.LOCA_OP_ERROR_TARGETS, nb, n_mb, d, k, cfg.C, r_a, nl, self.acc),
            loca.workspace_size(loca.LOCA_OP_ACCUMULATE_STATS, nb, n_mb, d, k, cfg.C, r_a, nl, self.acc),
            loca.workspace_size(loca.LOCA_OP_RIDGE_SOLVE, nb, n_mb, d, kp, cfg.C, r_a, nl, self.acc),
            loca.workspace_size(loca.LOCA_OP_LOWRANK_TRUNCATE, nb * nl, n_mb, d, kp, cfg.C, r_a, nl, self.acc),
        )
        self.ws = loca.alloc_workspace(ws, device)
        if poison:
            # NaN in every output (S and K too: the first micro-batch overwrites them, and
            # the entries of S below the diagonal are never read) and all-ones bytes in the
            # workspaces, so that a region a call should write but does not shows up as NaN
            for t in (self.Y, self.M, self.A_ad, self.B_ad, self.sigma, self.S, self.K) + \
                    ((self.B_proj,) if projected else ()):
                t.fill_(float("nan"))
            self.ws.fill_(255)
            if projected:
                self.ws_proj.fill_(255)

    @property
    def info(self):
        """Every dev_info slice of the step, concatenated (device int32; all zero when no
        call reported a condition)."""
        import torch
        return torch.cat([self.info_err, self.info_stats.reshape(-1), self.info_solve, self.info_trunc,
                          self.info_proj])

    def reset(self):
        # the first micro-batch's call overwrites S and K: no clearing pass
        self.mb_log = []
        self._m = 0  # every call rewrites its own dev_info slice
        self._gram = False  # B~ B~^T not yet formed in this step

    def resume(self, S, K, m_done: int):
        """Continue a step from saved statistics (checkpoint and resume): S, K as they were
        after the step's first m_done micro-batches (1 <= m_done < n_micro); the next
        micro_batch call is micro-batch m_done and adds into them."""
        if not 1 <= m_done < self.cfg.n_micro:
            raise ValueError(f"m_done must lie in [1, {self.cfg.n_micro}), got {m_done}")
        self.S.copy_(S)
        self.K.copy_(K)
        self.mb_log = []
        self._m = m_done
        self._gram = False

    def micro_batch(self, x_m, logits_m, labels_m, credit_a, credit_b, keep_log=False, stream=None, w=None, a=None):
        """Rows a1-a4 for one micro-batch: x_m (nb, n_m, d); w (n_m,) optional loss weights;
        a (n_m,) optional statistic weights (Section S7's weighted statistics)."""
        n_m = x_m.shape[1]
        y = self.Y[:, :n_m]
        m = self._m
        if m >= self.cfg.n_micro:
            raise ValueError(f"more than {self.cfg.n_micro} micro-batches since reset()")
        self._m += 1
        if not self._gram:  # B~ is fixed for the step: its Gram serves every micro-batch
            loca.loca_credit_gram(credit_b, self.G, self.ws, stream=stream)
            self._gram = True
        loca.loca_error_targets(logits_m, labels_m, credit_a, credit_b, y, self.mb, self.info_err[m:m + 1], self.ws,
                                w=w, a_w=a, nb=self.nb, credit_gram=self.G, stream=stream)
        loca.loca_accumulate_stats(x_m, y, self.cfg.eta, self.mb, self.S, self.K, self.ws, a_w=a,
                                   dev_info=self.info_stats[m], overwrite=m == 0, stream=stream)
        if keep_log:
            self.mb_log.append(self.mb.clone())

    def solve(self, credit_b, proj_a=None, stream=None, lp=None, rp=None, mid_event=None, trunc_event=None):
        """Rows a5-a6: ridge solves for every lambda and the rank-r_a truncation.

        With a current adapter W_prev = Lp Rp (lp: (nb, d, r_prev), rp: (nb, r_prev, d);
        the outer iteration past its first step, Theorem S6.1 with W_prev != 0), the solve
        takes the right-hand sides [S Lp | K] and W = M [Rp; B~] is truncated from its
        factors; the stacked right factor is a copy (layout only).  The projected solve
        (with proj_a) needs only the statistics: it is issued first, on the side stream
        after the statistics, and the current stream waits for it after the truncation.
        mid_event, when given, is recorded on the current stream between the solves and the
        truncation, and trunc_event after the truncation (before that wait)."""
        import torch
        cfg = self.cfg
        nl = len(cfg.lambdas)
        kp = self.r_prev + cfg.k
        cur = stream if stream is not None else torch.cuda.current_stream()
        side = self.projected and proj_a is not None
        if side:
            self.side.wait_stream(cur)  # the statistics have landed
            loca.loca_ridge_solve_projected(self.S, self.K, credit_b, proj_a, cfg.lambdas, self.B_proj,
                                            self.info_proj, self.ws_proj, stream=self.side)
        if self.r_prev > 0:
            assert lp is not None and rp is not None and lp.shape[-1] == self.r_prev
            loca.loca_ridge_solve(self.S, self.K, cfg.lambdas, self.M, self.info_solve, self.ws, lp=lp, rp=rp,
                                  stream=stream)
            right = torch.cat([rp, credit_b], dim=1).contiguous()
        else:
            loca.loca_ridge_solve(self.S, self.K, cfg.lambdas, self.M, self.info_solve, self.ws, stream=stream)
            right = credit_b
        if mid_event is not None:
            mid_event.record(cur)
        loca.loca_lowrank_truncate(self.M.view(self.nb * nl, cfg.d, kp), right, cfg.r_a, self.A_ad, self.B_ad,
                                   self.sigma, self.info_trunc, self.ws, r_group=nl, stream=stream)
        if trunc_event is not None:
            trunc_event.record(cur)
        if side:
            cur.wait_stream(self.side)

    def run(self, x_blocks, logits, labels, credit_a, credit_b, proj_a=None, stream=None, lp=None, rp=None):
        """One full pass over all micro-batches of all nb blocks (with the current adapter
        W_prev = lp rp when given)."""
        self.reset()
        for m in range(self.cfg.n_micro):
            lo, hi = self.cfg.micro_rows(m)
            self.micro_batch(x_blocks[:, lo:hi], logits[lo:hi], labels[lo:hi], credit_a, credit_b, stream=stream)
        self.solve(credit_b, proj_a, stream=stream, lp=lp, rp=rp)


class JacobiOuterLoop:
    """The outer iteration with the Jacobi schedule (Section S8): the caller runs one
    forward pass of the adapted model and passes every block's inputs and the shared
    logits to update(); each block then takes its step from that same forward pass with
    the residual target of its current adapter W_prev = Lp Rp (Eq. 6, Theorem S6.1), and
    the rank-r_a truncation of its solution becomes its next current adapter.  The first
    update starts from the frozen model (Lp = Rp = 0).  Orchestration only: every step runs
    in libloca's kernels; the factor transposes are layout copies."""

    def __init__(self, cfg: LocaConfig, nb: int, device="cuda"):
        import torch
        if len(cfg.lambdas) != 1:
            raise ValueError("the outer iteration keeps one adapter per block: give one lambda")
        self.cfg, self.nb = cfg, nb
        self.step = BlockStep(cfg, nb, device, r_prev=cfg.r_a)
        self.lp = torch.zeros((nb, cfg.d, cfg.r_a), dtype=torch.float32, device=device)
        self.rp = torch.zeros((nb, cfg.r_a, cfg.d), dtype=torch.float32, device=device)

    def adapters(self):
        """Current adapters as factors (Lp (nb, d, r_a), Rp (nb, r_a, d)): W_l = Lp_l Rp_l."""
        return self.lp, self.rp

    def update(self, x_blocks, logits, labels, credit_a, credit_b, stream=None):
        self.step.run(x_blocks, logits, labels, credit_a, credit_b, stream=stream, lp=self.lp, rp=self.rp)
        # W_r = A^T B^T with A (r_a x d), B (d x r_a): Lp = A^T, Rp = B^T
        self.lp.copy_(self.step.A_ad.transpose(1, 2))
        self.rp.copy_(self.step.B_ad.transpose(1, 2))
