"""Shared helpers of the test-suite: workload construction for both sides and
the oracle replay of a plan exported from the GPU."""
from __future__ import annotations

import numpy as np

from paper_2608_18484_amd import workloads as W


def rel_l2(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def params_for(wl: W.Workload, **over):
    from paper_2608_18484_amd import sparsepr as S
    ck, cq = wl.groups()
    kw = dict(n_sampled_queries=wl.n_sampled, r_k=wl.r_k, r_q=wl.r_q, n_kv_groups=ck,
              n_q_groups=cq, kmeans_iters=wl.kmeans_iters, target_exec_density=wl.density,
              n_probes=wl.n_probes, resid_rank=wl.resid_rank, ridge=wl.ridge,
              n_dense_prefix=wl.n_text)
    kw.update(over)
    return S.default_params(**kw)


def oracle_kwargs(p):
    """Oracle arguments equal to a Params struct (density as the float the GPU sees)."""
    return dict(n_text=p.n_dense_prefix, n_sampled=p.n_sampled_queries, r_k=p.r_k, r_q=p.r_q,
                c_k=p.n_kv_groups, c_q=p.n_q_groups, iters=p.kmeans_iters,
                density=float(np.float32(p.target_exec_density)), n_probes=p.n_probes,
                r=p.resid_rank, lam=float(np.float32(p.ridge)), partition=p.partition,
                probe_rule=p.probe_rule, probe_seed=p.probe_seed, ridge_only=p.ridge_only,
                routing=p.routing)


def to_device(q, k, v, dtype):
    import torch
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    return tuple(torch.from_numpy(np.ascontiguousarray(x)).to("cuda").to(tdt) for x in (q, k, v))


def medium(grid=(4, 24, 32), heads=2, dtype="bf16", d=128, **kw):
    """A workload the oracle finishes in seconds that still spans many tiles."""
    base = dict(length_scale=None, length_range=(2.0, 6.0), n_sampled=256, density=0.25,
                n_probes=64, resid_rank=16, ridge=0.1)
    base.update(kw)
    return W.Workload("medium", 1, heads, grid, d, dtype, **base)
