"""Seeded synthetic attention inputs shaped like video-token workloads.

This module only draws inputs. It holds none of the operator's arithmetic and
is the one piece shared by the CPU oracle's tests and the GPU path, so both
sides see byte-identical Q, K and V.

Inputs stand in for real activations of video diffusion / world models (the
paper measures on real models, Sec. 5): tokens sit on a (T, H, W) grid in
raster order, token n = (t*H + y)*W + x, and every head draws

    phi_j(p) = sqrt(2) * cos(omega_j . p + b_j),  j = 1..64,
    omega_j ~ N(0, l^-2 I_3),  b_j ~ U[0, 2 pi)
    W in R^{d x 64}, W_ij ~ N(0, 1/64)            (shared by Q, K and V)
    Q = beta * (W phi + sigma_q eps_Q),  K = W phi + sigma eps_K,  V = W phi + sigma eps_V

so q.k is a random-Fourier-feature estimate of an RBF kernel of the position
difference and attention is spatiotemporally local.  Each (batch, head) uses
numpy.random.default_rng([seed, b, h]) and draws, in this order: the length
scale l_h, Omega, the phases b, W, eps_Q, eps_K, eps_V (text tokens, where
present, are drawn after those).  Data is generated in float32; the bf16
configurations are rounded to bf16 (round-to-nearest-even) by the caller, and
both the oracle and the GPU read the rounded values.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional

import numpy as np

N_FEAT = 64


@dataclasses.dataclass(frozen=True)
class Workload:
    """One attention-layer workload: grid, heads, generator and method knobs."""

    name: str
    batch: int
    heads: int
    grid: tuple  # (T, H, W) video grid
    d: int
    dtype: str  # "f32" or "bf16"
    # generator
    length_scale: Optional[float] = None  # fixed l; None -> l_h ~ U[lo, hi]
    length_range: tuple = (2.0, 8.0)
    sigma: float = 0.3
    sigma_q: float = 0.3
    beta: float = 1.0
    tune_tau: Optional[float] = None  # target median tau(0.9); None -> fixed beta
    n_text: int = 0  # i.i.d. N(0,1) text tokens prepended to the grid
    cond_frames: int = 0  # leading frames drawn with their own generator
    cond_length: float = 1.5
    cond_sigma: float = 0.1
    seed: int = 0
    # method parameters
    n_sampled: int = 256
    n_kv_groups: int = 0  # 0 -> ceil(N_video / 64)
    n_q_groups: int = 0
    density: float = 0.25
    n_probes: int = 128
    resid_rank: int = 16
    ridge: float = 0.1
    r_k: int = 48
    r_q: int = 64
    kmeans_iters: int = 8

    @property
    def n_video(self) -> int:
        t, h, w = self.grid
        return t * h * w

    @property
    def n(self) -> int:
        return self.n_video + self.n_text

    def groups(self):
        ck = self.n_kv_groups or -(-self.n_video // 64)
        cq = self.n_q_groups or -(-self.n_video // 64)
        return ck, cq

    def with_(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


# The five workload families (tiny fp32 check, video DiT layer, long video,
# text + video joint attention, two-branch world model).
CONFIGS = {
    "tiny": Workload("tiny", 1, 1, (4, 16, 16), 64, "f32", length_scale=4.0,
                     n_sampled=64, n_kv_groups=16, n_q_groups=16, density=0.25,
                     n_probes=32, resid_rank=8, ridge=1e-4),
    "video_dit": Workload("video_dit", 1, 24, (11, 30, 52), 128, "bf16"),
    "long_video": Workload("long_video", 1, 24, (21, 45, 80), 128, "bf16", tune_tau=0.06),
    "text_video": Workload("text_video", 1, 24, (33, 45, 80), 128, "bf16", tune_tau=0.06,
                           n_text=256, n_probes=192),
    "world_model": Workload("world_model", 2, 16, (24, 44, 80), 128, "bf16",
                            length_range=(3.0, 8.0), sigma=0.5, sigma_q=0.5,
                            cond_frames=4, cond_length=1.5, cond_sigma=0.1),
}


def grid_positions(grid) -> np.ndarray:
    t, h, w = grid
    tt, yy, xx = np.meshgrid(np.arange(t), np.arange(h), np.arange(w), indexing="ij")
    return np.stack([tt.ravel(), yy.ravel(), xx.ravel()], axis=1).astype(np.float64)


def _features(rng, pos, length):
    omega = rng.standard_normal((N_FEAT, 3)) / length
    phase = rng.uniform(0.0, 2.0 * math.pi, N_FEAT)
    return (math.sqrt(2.0) * np.cos(pos @ omega.T + phase)).astype(np.float32)


def _tau90_median(q0, k, n_rows=32, mass=0.9):
    """Median over strided rows of the fraction of keys holding `mass` of the
    row's softmax mass, as a function of the query scale beta (returned as a
    callable).  Used only to shape the synthetic workload."""
    n = q0.shape[0]
    rows = (np.arange(n_rows) * n) // n_rows
    logits = (q0[rows].astype(np.float64) @ k.T.astype(np.float64)) / math.sqrt(k.shape[1])
    srt = -np.sort(-logits, axis=1)
    top = srt[:, :1]
    nk = k.shape[0]

    def tau(beta):
        p = np.exp(beta * (srt - top))
        c = np.cumsum(p, axis=1)
        need = mass * c[:, -1:]
        cnt = (c < need).sum(axis=1) + 1
        return float(np.median(cnt / nk))

    return tau


def _tune_beta(q0, k, target):
    tau = _tau90_median(q0, k)
    lo, hi = math.log(0.05), math.log(8.0)
    for _ in range(22):
        mid = 0.5 * (lo + hi)
        if tau(math.exp(mid)) > target:
            lo = mid  # too broad -> sharpen
        else:
            hi = mid
    beta = math.exp(0.5 * (lo + hi))
    return float(f"{beta:.3g}")


def make_head(wl: Workload, b: int, h: int):
    """Draw (q, k, v, beta, l) for one (batch, head) as float32 [N, d]."""
    rng = np.random.default_rng([wl.seed, b, h])
    lo, hi = wl.length_range
    l_draw = rng.uniform(lo, hi)
    length = wl.length_scale if wl.length_scale is not None else l_draw
    pos = grid_positions(wl.grid)
    nv, d = wl.n_video, wl.d
    feats = _features(rng, pos, length)
    w = (rng.standard_normal((d, N_FEAT)) / math.sqrt(N_FEAT)).astype(np.float32)
    sig = np.full((nv, 1), wl.sigma, np.float32)
    sig_q = np.full((nv, 1), wl.sigma_q, np.float32)
    if wl.cond_frames:
        t, hh, ww = wl.grid
        nc = wl.cond_frames * hh * ww
        feats[:nc] = _features(rng, pos[:nc], wl.cond_length)
        sig[:nc] = wl.cond_sigma
        sig_q[:nc] = wl.cond_sigma
    signal = feats @ w.T
    eq = rng.standard_normal((nv, d), dtype=np.float32)
    ek = rng.standard_normal((nv, d), dtype=np.float32)
    ev = rng.standard_normal((nv, d), dtype=np.float32)
    q0 = signal + sig_q * eq
    k = signal + sig * ek
    v = signal + sig * ev
    beta = wl.beta
    if wl.tune_tau is not None:
        beta = _tune_beta(q0, k, wl.tune_tau)
    q = (beta * q0).astype(np.float32)
    if wl.n_text:
        tq = rng.standard_normal((wl.n_text, d), dtype=np.float32)
        tk = rng.standard_normal((wl.n_text, d), dtype=np.float32)
        tv = rng.standard_normal((wl.n_text, d), dtype=np.float32)
        q = np.concatenate([tq, q])
        k = np.concatenate([tk, k])
        v = np.concatenate([tv, v])
    return q, k.astype(np.float32), v.astype(np.float32), beta, length


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round float32 to the nearest bfloat16 (ties to even), returned as float32."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = ((u >> 16) & 1) + np.uint32(0x7FFF)
    return ((u + r) & np.uint32(0xFFFF0000)).view(np.float32)


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """The uint16 bit patterns of bf16_round(x)."""
    return (bf16_round(x).view(np.uint32) >> 16).astype(np.uint16)


def make_inputs(wl: Workload, heads: Optional[list] = None, workers: int = 1):
    """Q, K, V as float32 [B, H, N, d] (already rounded to bf16 values when
    wl.dtype == 'bf16'), plus per-head generator metadata.  `heads` limits
    generation to a list of (b, h) pairs; other heads are left at zero.
    `workers` > 1 draws heads on a thread pool (each head has its own
    generator, so the result does not depend on it)."""
    shape = (wl.batch, wl.heads, wl.n, wl.d)
    q = np.zeros(shape, np.float32)
    k = np.zeros(shape, np.float32)
    v = np.zeros(shape, np.float32)
    meta = {}
    todo = heads if heads is not None else [(b, h) for b in range(wl.batch) for h in range(wl.heads)]

    def one(bh):
        b, h = bh
        qh, kh, vh, beta, length = make_head(wl, b, h)
        if wl.dtype == "bf16":
            qh, kh, vh = bf16_round(qh), bf16_round(kh), bf16_round(vh)
        q[b, h], k[b, h], v[b, h] = qh, kh, vh
        return bh, {"beta": beta, "length": length}

    if workers > 1:
        from concurrent.futures import ThreadPoolExecutor
        with ThreadPoolExecutor(workers) as ex:
            for bh, m in ex.map(one, todo):
                meta[bh] = m
    else:
        for bh in todo:
            meta[bh] = one(bh)[1]
    return q, k, v, meta


def strided_rows(n: int, m: int) -> np.ndarray:
    """m rows spread evenly over [0, n)."""
    m = min(m, n)
    return ((np.arange(m, dtype=np.int64) * n) // m).astype(np.int64)
