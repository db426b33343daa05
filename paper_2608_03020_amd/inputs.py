"""Seeded synthetic inputs for the LoCA per-block adaptation step.

This module only draws random numbers and lays them out; it holds none of the
method's arithmetic (no softmax, no statistics, no solve).  It is the one piece
shared by the float64 oracle's tests and the HIP path's callers.

The workloads stand in for Qwen2.5 forward activations on the paper's tasks
(Section "Experiments -- Setup"; datasets and checkpoints are not available):
Qwen2.5-shaped widths and block counts, small label sets like the tasks' answer
sets, and the full 151,936-token vocabulary for the full-vocabulary variant.

Two backends follow the same recipe:
  * ``numpy``  -- host arrays, SFC64 streams keyed by (seed, config, block,
    tensor, micro-batch); used by CPU tests, GPU parity tests and the CPU
    baseline sample.
  * ``torch``  -- device tensors from a seeded ``torch.Generator`` on the GPU;
    used where the full workload is too large to draw on the host (the bench,
    full-size sampled parity).  Values differ from the numpy backend; the
    distributions are the same.

bf16 values are produced by round-to-nearest-even from float32.
"""
from __future__ import annotations

import dataclasses
from typing import Optional, Tuple

import numpy as np

# ---------------------------------------------------------------- config table


@dataclasses.dataclass(frozen=True)
class LocaConfig:
    name: str
    blocks: int          # L, transformer blocks (independent under the Jacobi schedule)
    d: int               # hidden width
    n: int               # selected prediction positions per block solve
    micro: int           # tokens per micro-batch (each has its own eta_bar)
    C: int               # classes of the error softmax (label set, or vocabulary)
    k: int               # credit rank of the fixed feedback factors
    r_a: int             # adapter rank
    lambdas: Tuple[float, ...]
    mode: str            # "fp32": fp32 inputs, fp64 statistics; "bf16": bf16 X, fp32 statistics
    x_dist: str          # "gauss_outlier" | "rms_outlier" | "student_t"
    n_outlier: int       # outlier channels (gauss_outlier / rms_outlier)
    outlier_scale: float
    logit_std: float
    logit_dtype: str     # "f32" | "bf16"
    a_dtype: str         # dtype of the credit factor A~ (C x k): "f32" | "bf16"
    eta: float = 0.01    # dimensionless target size (middle of the candidate set {0.003, 0.01, 0.03})

    @property
    def n_micro(self) -> int:
        return (self.n + self.micro - 1) // self.micro

    def micro_rows(self, m: int) -> Tuple[int, int]:
        lo = m * self.micro
        return lo, min(self.n, lo + self.micro)


CONFIGS = {
    # Single block, Qwen2.5-0.5B width, fp32 mode.
    "c1": LocaConfig("c1", 1, 896, 512, 512, 2, 8, 8, (1e-2,), "fp32",
                     "gauss_outlier", 4, 20.0, 2.0, "f32", "f32"),
    # Qwen2.5-1.5B-shaped, 4 micro-batches of 2048.
    "c2": LocaConfig("c2", 28, 1536, 8192, 2048, 4, 16, 16, (1e-2,), "bf16",
                     "rms_outlier", 8, 30.0, 3.0, "f32", "f32"),
    # Qwen2.5-7B-shaped, three ridge strengths solved from the same statistics.
    "c3": LocaConfig("c3", 28, 3584, 32768, 8192, 5, 32, 16, (1e-3, 1e-2, 1e-1), "bf16",
                     "rms_outlier", 18, 30.0, 3.0, "f32", "f32"),
    # Full-vocabulary error variant, Qwen2.5-3B width.
    "c4": LocaConfig("c4", 1, 2048, 4096, 4096, 151936, 64, 32, (1e-2,), "bf16",
                     "rms_outlier", 10, 30.0, 2.0, "bf16", "bf16"),
    # Qwen2.5-14B-shaped, heavy-tailed activations, 8 chunks of 8192.
    "c5": LocaConfig("c5", 48, 5120, 65536, 8192, 5, 64, 32, (1e-2,), "bf16",
                     "student_t", 0, 1.0, 3.0, "f32", "f32"),
}

_CFG_ID = {"c1": 1, "c2": 2, "c3": 3, "c4": 4, "c5": 5}
# tensor ids inside a (config, block) key
(_T_X, _T_LOGITS, _T_LABELS, _T_A, _T_B, _T_OUTL, _T_SCALE, _T_ADAPT, _T_CURRENT, _T_WEIGHTS, _T_PROBE,
 _T_STATW, _T_LINNET) = range(13)


def custom_config(name="tiny", blocks=1, d=64, n=100, micro=None, C=5, k=8, r_a=4,
                  lambdas=(1e-2,), mode="bf16", x_dist="rms_outlier", n_outlier=2,
                  outlier_scale=30.0, logit_std=3.0, logit_dtype="f32", a_dtype="f32",
                  eta=0.01) -> LocaConfig:
    return LocaConfig(name, blocks, d, n, micro or n, C, k, r_a, tuple(lambdas), mode,
                      x_dist, n_outlier, outlier_scale, logit_std, logit_dtype, a_dtype, eta)


# ---------------------------------------------------------------- bf16 helpers


def bf16_bits(a: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns (uint16), round to nearest even."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_to_f32(h: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(h, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


# ---------------------------------------------------------------- numpy backend


def _rng(seed: int, cfg: LocaConfig, block: int, tensor: int, micro: int = 0) -> np.random.Generator:
    cid = _CFG_ID.get(cfg.name, 99)
    ss = np.random.SeedSequence([seed, cid, block, tensor, micro, cfg.d, cfg.C, cfg.k])
    return np.random.Generator(np.random.SFC64(ss))


def outlier_channels(cfg: LocaConfig, block: int, seed: int = 0) -> np.ndarray:
    if cfg.n_outlier <= 0:
        return np.zeros(0, dtype=np.int64)
    g = _rng(seed, cfg, block, _T_OUTL)
    return np.sort(g.choice(cfg.d, size=min(cfg.n_outlier, cfg.d), replace=False))


def channel_scales(cfg: LocaConfig, block: int, seed: int = 0) -> np.ndarray:
    """Per-channel log-normal scales (sigma = 1) of the heavy-tailed recipe."""
    g = _rng(seed, cfg, block, _T_SCALE)
    return np.exp(g.standard_normal(cfg.d)).astype(np.float32)


def gen_x(cfg: LocaConfig, block: int, m: int, seed: int = 0) -> np.ndarray:
    """Block input X for micro-batch m, token-major (rows x d).

    Returns float32 for fp32 mode, bf16 bit patterns (uint16) for bf16 mode.
    """
    lo, hi = cfg.micro_rows(m)
    rows = hi - lo
    g = _rng(seed, cfg, block, _T_X, m)
    if cfg.x_dist == "gauss_outlier":
        x = g.standard_normal((rows, cfg.d), dtype=np.float32)
        x[:, outlier_channels(cfg, block, seed)] *= np.float32(cfg.outlier_scale)
    elif cfg.x_dist == "rms_outlier":
        x = g.standard_normal((rows, cfg.d), dtype=np.float32)
        x /= np.sqrt(np.mean(x.astype(np.float64) ** 2, axis=1, keepdims=True)).astype(np.float32)
        x[:, outlier_channels(cfg, block, seed)] *= np.float32(cfg.outlier_scale)
    elif cfg.x_dist == "student_t":
        x = g.standard_t(4.0, size=(rows, cfg.d)).astype(np.float32)
        x *= channel_scales(cfg, block, seed)[None, :]
    else:
        raise ValueError(cfg.x_dist)
    if cfg.mode == "fp32":
        return np.ascontiguousarray(x, dtype=np.float32)
    return bf16_bits(x)


def gen_logits(cfg: LocaConfig, m: int, seed: int = 0) -> np.ndarray:
    """Frozen-head logits for micro-batch m (rows x C); shared by all blocks."""
    lo, hi = cfg.micro_rows(m)
    g = _rng(seed, cfg, 0, _T_LOGITS, m)
    z = (g.standard_normal((hi - lo, cfg.C), dtype=np.float32) * np.float32(cfg.logit_std))
    return z if cfg.logit_dtype == "f32" else bf16_bits(z)


def gen_labels(cfg: LocaConfig, m: int, seed: int = 0) -> np.ndarray:
    lo, hi = cfg.micro_rows(m)
    g = _rng(seed, cfg, 0, _T_LABELS, m)
    return g.integers(0, cfg.C, size=hi - lo, dtype=np.int32)


def gen_credit(cfg: LocaConfig, block: int, seed: int = 0):
    """Per-block credit factors (A~: C x k, B~: k x d), entries ~ N(0, 1/k)."""
    s = np.float32(1.0 / np.sqrt(cfg.k))
    a = _rng(seed, cfg, block, _T_A).standard_normal((cfg.C, cfg.k), dtype=np.float32) * s
    b = _rng(seed, cfg, block, _T_B).standard_normal((cfg.k, cfg.d), dtype=np.float32) * s
    if cfg.a_dtype == "bf16":
        a = bf16_bits(a)
    return a, b


def gen_adapter_projection(cfg: LocaConfig, block: int, seed: int = 0) -> np.ndarray:
    """Fixed random adapter projection A_l (r_a x d), entries ~ N(0, 1/d)."""
    g = _rng(seed, cfg, block, _T_ADAPT)
    return g.standard_normal((cfg.r_a, cfg.d), dtype=np.float32) * np.float32(1.0 / np.sqrt(cfg.d))


def gen_current_adapter(cfg: LocaConfig, block: int, r_prev: int, seed: int = 0):
    """A current adapter W_prev = Lp Rp of rank r_prev in factored form (float32):
    Lp (d x r_prev) with orthonormal-ish columns ~ N(0, 1/d), Rp (r_prev x d) ~ N(0, 1/d).
    Callers rescale Rp to the scale they need."""
    g = _rng(seed, cfg, block, _T_CURRENT)
    lp = g.standard_normal((cfg.d, r_prev), dtype=np.float32) * np.float32(1.0 / np.sqrt(cfg.d))
    rp = g.standard_normal((r_prev, cfg.d), dtype=np.float32) * np.float32(1.0 / np.sqrt(cfg.d))
    return lp, rp


def gen_loss_weights(cfg: LocaConfig, micro: int, masked: float = 0.2, seed: int = 0) -> np.ndarray:
    """Per-position loss weights w_t >= 0 of micro-batch `micro` (float32): uniform on
    [0, 2), with a fraction `masked` of positions set to 0 (masked positions)."""
    g = _rng(seed, cfg, 0, _T_WEIGHTS, micro)
    lo, hi = cfg.micro_rows(micro)
    w = (2.0 * g.random(hi - lo)).astype(np.float32)
    w[g.random(hi - lo) < masked] = 0.0
    return w


def gen_stat_weights(cfg: LocaConfig, micro: int, zero: float = 0.2, seed: int = 0) -> np.ndarray:
    """Per-position statistic weights a_t >= 0 of micro-batch `micro` (float32):
    uniform on [0, 2) with a fraction `zero` of positions at 0 (dropped positions)."""
    g = _rng(seed, cfg, 0, _T_STATW, micro)
    lo, hi = cfg.micro_rows(micro)
    a = (2.0 * g.random(hi - lo)).astype(np.float32)
    a[g.random(hi - lo) < zero] = 0.0
    return a


def gen_probe_pairs(cfg: LocaConfig, n_p: int, blocks: int, rank: int = 0, noise: float = 2.0, seed: int = 0):
    """Synthetic calibration probes (float32): top errors E (d x n_p) ~ N(0, 1) shared by
    the blocks, and per block gradients G_b = F0_b E + noise * N(0, 1) with a seeded
    rank-`rank` map F0_b = P_b Q_b^T (P, Q ~ N(0, 1/d); rank 0 means 2k).  The noise
    level sets how far a fitted map can align with G (the paper reports 0.3-0.5)."""
    g = _rng(seed, cfg, 0, _T_PROBE)
    E = g.standard_normal((cfg.d, n_p), dtype=np.float32)
    r = rank or 2 * cfg.k
    Gs = []
    for b in range(blocks):
        gb = _rng(seed, cfg, b, _T_PROBE, 1)
        P = gb.standard_normal((cfg.d, r), dtype=np.float32) / np.float32(np.sqrt(cfg.d))
        Q = gb.standard_normal((cfg.d, r), dtype=np.float32) / np.float32(np.sqrt(cfg.d))
        Gs.append((P @ (Q.T @ E) + np.float32(noise / np.sqrt(cfg.d)) * gb.standard_normal((cfg.d, n_p),
                                                                                             dtype=np.float32))
                  .astype(np.float32))
    return E, np.stack(Gs)


def gen_linear_network(cfg: LocaConfig, seed: int = 0, mix: float = 0.5):
    """A synthetic network of cfg.blocks linear residual blocks, the frozen-backbone
    stand-in of the outer-iteration tests: token features h0 (n x d, N(0,1)), block maps
    F_l (d x d, N(0, mix^2/d)) with h_l = h_{l-1} (I + F_l), a head W_u (C x d, N(0, 4/d))
    and labels.  float32 values (exact in float64 as well)."""
    g = _rng(seed, cfg, 0, _T_LINNET)
    n, d, L, C = cfg.n, cfg.d, cfg.blocks, cfg.C
    h0 = g.standard_normal((n, d), dtype=np.float32)
    Fs = g.standard_normal((L, d, d), dtype=np.float32) * np.float32(mix / np.sqrt(d))
    Wu = g.standard_normal((C, d), dtype=np.float32) * np.float32(2.0 / np.sqrt(d))
    y = g.integers(0, C, n).astype(np.int32)
    return h0, Fs, Wu, y


def as_f64(a: np.ndarray, dtype: str) -> np.ndarray:
    """Exact float64 value of a generated array (bf16 bit patterns or float32)."""
    if dtype == "bf16" or a.dtype == np.uint16:
        return bf16_to_f32(a).astype(np.float64)
    return np.asarray(a, dtype=np.float64)


# ---------------------------------------------------------------- torch device backend


def torch_gen_x(cfg: LocaConfig, rows: int, generator, device="cuda", outliers=None, scales=None):
    """Device-side X with the recipe of ``gen_x`` (values differ from numpy's)."""
    import torch
    x = torch.randn((rows, cfg.d), generator=generator, device=device, dtype=torch.float32)
    if cfg.x_dist == "gauss_outlier":
        if outliers is not None and len(outliers):
            x[:, outliers] *= cfg.outlier_scale
    elif cfg.x_dist == "rms_outlier":
        x /= x.square().mean(dim=1, keepdim=True).sqrt()
        if outliers is not None and len(outliers):
            x[:, outliers] *= cfg.outlier_scale
    elif cfg.x_dist == "student_t":
        # Student-t(4) = N(0,1) / sqrt(chi2_4 / 4), chi2_4 = -2 log(U1 U2)
        u = torch.rand((2, rows, cfg.d), generator=generator, device=device, dtype=torch.float32)
        u = u.clamp_min_(1e-30)
        chi2 = -2.0 * (u[0].log() + u[1].log())
        x /= (chi2 / 4.0).sqrt()
        del u, chi2
        if scales is not None:
            x *= scales[None, :]
    if cfg.mode == "fp32":
        return x
    return x.to(torch.bfloat16)


def torch_gen_block_inputs(cfg: LocaConfig, block: int, seed: int = 0, device="cuda",
                           rows: Optional[int] = None):
    """Device X (all micro-batches, rows x d) for one block plus its credit factors."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed((seed * 1000003 + _CFG_ID.get(cfg.name, 99) * 7919 + block) & 0x7FFFFFFF)
    outl = torch.as_tensor(outlier_channels(cfg, block, seed), device=device)
    scales = torch.as_tensor(channel_scales(cfg, block, seed), device=device) if cfg.x_dist == "student_t" else None
    x = torch_gen_x(cfg, rows or cfg.n, g, device, outl, scales)
    a, b = gen_credit(cfg, block, seed)
    ta = torch.as_tensor(a.view(np.int16) if a.dtype == np.uint16 else a, device=device)
    if a.dtype == np.uint16:
        ta = ta.view(torch.bfloat16)
    return x, ta, torch.as_tensor(b, device=device)


def torch_gen_head(cfg: LocaConfig, seed: int = 0, device="cuda", rows: Optional[int] = None):
    """Device logits (rows x C) and labels (rows) with the recipe of gen_logits / gen_labels."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed((seed * 1000003 + _CFG_ID.get(cfg.name, 99) * 7919 + 104729) & 0x7FFFFFFF)
    rows = rows or cfg.n
    z = torch.randn((rows, cfg.C), generator=g, device=device, dtype=torch.float32) * cfg.logit_std
    if cfg.logit_dtype == "bf16":
        z = z.to(torch.bfloat16)
    y = torch.randint(0, cfg.C, (rows,), generator=g, device=device, dtype=torch.int32)
    return z, y


def torch_gen_stat_weights(cfg: LocaConfig, seed: int = 0, device="cuda", zero: float = 0.2):
    """Device statistic weights for all cfg.n positions, with the recipe of gen_stat_weights."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed((seed * 1000003 + _CFG_ID.get(cfg.name, 99) * 7919 + 15485863) & 0x7FFFFFFF)
    a = 2.0 * torch.rand(cfg.n, generator=g, device=device, dtype=torch.float32)
    a[torch.rand(cfg.n, generator=g, device=device) < zero] = 0.0
    return a


def torch_gen_adapter_projection(cfg: LocaConfig, blocks: int, seed: int = 0, device="cuda"):
    """Device projections A_l (blocks, r_a, d) of the projected form, with the recipe of
    gen_adapter_projection (entries ~ N(0, 1/d))."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed((seed * 1000003 + _CFG_ID.get(cfg.name, 99) * 7919 + 67867967) & 0x7FFFFFFF)
    return torch.randn((blocks, cfg.r_a, cfg.d), generator=g, device=device, dtype=torch.float32) / np.sqrt(cfg.d)


def torch_gen_current_adapter(cfg: LocaConfig, blocks: int, r_prev: int, seed: int = 0, device="cuda"):
    """Device current adapters W_prev = Lp Rp of every block, with the recipe of
    gen_current_adapter: Lp (blocks, d, r_prev), Rp (blocks, r_prev, d)."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed((seed * 1000003 + _CFG_ID.get(cfg.name, 99) * 7919 + 32452843) & 0x7FFFFFFF)
    s = 1.0 / np.sqrt(cfg.d)
    lp = torch.randn((blocks, cfg.d, r_prev), generator=g, device=device, dtype=torch.float32) * s
    rp = torch.randn((blocks, r_prev, cfg.d), generator=g, device=device, dtype=torch.float32) * s
    return lp, rp


def torch_gen_probe_pairs(cfg: LocaConfig, n_p: int, blocks: int, seed: int = 0, device="cuda",
                          noise: float = 2.0):
    """Device calibration probes with the recipe of gen_probe_pairs (rank-2k maps):
    E (d, n_p) shared by the blocks and G (blocks, d, n_p)."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed((seed * 1000003 + _CFG_ID.get(cfg.name, 99) * 7919 + 49979687) & 0x7FFFFFFF)
    d, r = cfg.d, 2 * cfg.k
    E = torch.randn((d, n_p), generator=g, device=device, dtype=torch.float32)
    s = 1.0 / np.sqrt(d)
    P = torch.randn((blocks, d, r), generator=g, device=device, dtype=torch.float32) * s
    Q = torch.randn((blocks, d, r), generator=g, device=device, dtype=torch.float32) * s
    G = P @ (Q.transpose(1, 2) @ E) + (noise * s) * torch.randn((blocks, d, n_p), generator=g, device=device,
                                                                   dtype=torch.float32)
    return E, G.contiguous()
