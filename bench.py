#!/usr/bin/env python3
"""Benchmark of one SparsePR attention call (plan + attend over every head of
one layer) on the long-video workload: 24 heads, d = 128, bf16, a 21x45x80
token grid (N = 75,600), target executed-pair density 25 %.

Prints ONE JSON line: ms per call, effective TFLOP/s on executed pairs
(4 d per executed query-key pair), the output's error against dense attention,
the roofline of the dominant kernel (block-sparse attention, bf16 MFMA) timed
with HIP events on the stream it runs on, and the CPU oracle timed on one head
of the same workload on this host's cores (whole call extrapolated), plus an
fp64 dense cross-check of the dense reference on strided rows.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time
from concurrent.futures import ThreadPoolExecutor

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2608_18484_amd import workloads as W  # noqa: E402

BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 MFMA
# the attention kernel, and the planner that orders its chunks (dispatch
# order changes how much K/V is read again from beyond L2)
ATTN_SRCS = [os.path.join(ROOT, "paper_2608_18484_amd", "csrc", f)
             for f in ("attn_kernels.hip", "plan_kernels.hip")]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "k_attn_mfma_long_video_traffic.json")


def attn_traffic(workload):
    """HBM bytes of one call's sparse-attention launches, from the committed
    FETCH_SIZE / WRITE_SIZE counter runs (scaled by the copy calibration), or
    None when they were taken on another workload or on different kernel
    sources (attention and planner) than the ones built now."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
        h = hashlib.sha256()
        for src in ATTN_SRCS:
            with open(src, "rb") as f:
                h.update(f.read())
        sha = h.hexdigest()
    except (OSError, ValueError):
        return None
    if rec.get("source_sha256") != sha or rec.get("workload") != workload:
        return None
    return rec.get("hbm_bytes_per_call")


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def params_for(S, wl, density):
    ck, cq = wl.groups()
    return S.default_params(n_sampled_queries=wl.n_sampled, r_k=wl.r_k, r_q=wl.r_q,
                            n_kv_groups=ck, n_q_groups=cq, kmeans_iters=wl.kmeans_iters,
                            target_exec_density=density, n_probes=wl.n_probes,
                            resid_rank=wl.resid_rank, ridge=wl.ridge, n_dense_prefix=wl.n_text)


def generate(wl, torch):
    """Seeded inputs, generated per head on the host and placed in HBM as bf16."""
    shape = (wl.batch, wl.heads, wl.n, wl.d)
    tdt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    q = torch.empty(shape, dtype=tdt, device="cuda")
    k = torch.empty_like(q)
    v = torch.empty_like(q)
    host = {}

    def one(bh):
        b, h = divmod(bh, wl.heads)
        qh, kh, vh, _, _ = W.make_head(wl, b, h)
        if wl.dtype == "bf16":
            qh, kh, vh = W.bf16_round(qh), W.bf16_round(kh), W.bf16_round(vh)
        return bh, qh, kh, vh

    with ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as ex:
        for bh, qh, kh, vh in ex.map(one, range(wl.batch * wl.heads)):
            b, h = divmod(bh, wl.heads)
            for dst, src in ((q, qh), (k, kh), (v, vh)):
                dst[b, h].copy_(torch.from_numpy(src))
            if bh == 0:
                host = {"q": qh, "k": kh, "v": vh}
    torch.cuda.synchronize()
    return q, k, v, host


def head_inputs(wl, b, h):
    """Host copies of one head's inputs, exactly as placed in HBM."""
    qh, kh, vh, _, _ = W.make_head(wl, b, h)
    if wl.dtype == "bf16":
        qh, kh, vh = W.bf16_round(qh), W.bf16_round(kh), W.bf16_round(vh)
    return qh, kh, vh


def cpu_baseline(wl, host, density, n_heads=1):
    """The oracle, as it is, on the first `n_heads` heads of the same inputs:
    plan + attend, timed per head and summed; the whole call (all B*H heads)
    is extrapolated from the mean per head when fewer heads are timed."""
    import oracle
    oracle.build(force=False)
    ck, cq = wl.groups()
    n = wl.n
    total = wl.batch * wl.heads
    n_heads = max(1, min(n_heads, total))
    dt = 0.0
    exec_pairs = 0
    for bh in range(n_heads):
        b, h = divmod(bh, wl.heads)
        qh, kh, vh = (host["q"], host["k"], host["v"]) if bh == 0 else head_inputs(wl, b, h)
        t0 = time.perf_counter()
        out, pl = oracle.run(qh, kh, vh, n_text=wl.n_text,
                             n_sampled=wl.n_sampled, r_k=wl.r_k, r_q=wl.r_q, c_k=ck, c_q=cq,
                             iters=wl.kmeans_iters, density=float(np.float32(density)),
                             n_probes=wl.n_probes, r=wl.resid_rank, lam=float(np.float32(wl.ridge)))
        dt += time.perf_counter() - t0
        exec_pairs += int(pl["stats"][0]) + len(pl["probes"]) * n
        if n_heads > 1:
            log(f"CPU oracle: head {bh + 1}/{n_heads} done, {dt:.1f}s so far")
    flops = 4.0 * wl.d * exec_pairs
    per_call = dt / n_heads * total
    return {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": oracle.num_threads(),
            "kind": "oracle", "seconds": dt,
            "sample": f"{n_heads} of {total} heads (from b=0, h=0) at full size N={n}: "
                      f"plan + attend, {exec_pairs} executed pairs",
            "ms_per_call": round(per_call * 1e3, 1),
            "ms_per_call_kind": "measured (all heads)" if n_heads == total else
                                f"extrapolated: mean of {n_heads} head(s) x {total} heads"}


def dense_crosscheck(wl, host, dense_gpu, out_gpu, rows=1024):
    """fp64 dense attention of the oracle on `rows` strided rows of head (0, 0),
    against the GPU's dense reference (the MFMA kernel the error readout uses)
    and against the SparsePR output, on the same rows."""
    import oracle
    oracle.build(force=False)
    idx = W.strided_rows(wl.n, rows)
    ref = oracle.dense_rows(host["q"], host["k"], host["v"], idx)
    dg = dense_gpu[0, 0, idx].float().cpu().numpy().astype(np.float64)
    og = out_gpu[0, 0, idx].float().cpu().numpy().astype(np.float64)
    nrm = np.linalg.norm(ref)
    return {"rows": int(len(idx)), "head": [0, 0],
            "rel_l2_gpu_dense_vs_fp64": round(float(np.linalg.norm(dg - ref) / nrm), 8),
            "rel_l2_sparsepr_vs_fp64": round(float(np.linalg.norm(og - ref) / nrm), 6)}


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="long_video", choices=sorted(W.CONFIGS))
    ap.add_argument("--density", type=float, default=0.25)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-dense", action="store_true", help="skip the dense-attention error check")
    ap.add_argument("--cpu-heads", type=int, default=1,
                    help="heads the CPU oracle baseline runs (the whole call is extrapolated "
                         "from their mean when fewer than all)")
    ap.add_argument("--warm-start", action="store_true",
                    help="steady state of consecutive calls: both k-means start from the previous "
                         "call's centroids and run 2 assignments; calls alternate between the "
                         "inputs and a copy perturbed by 5%% noise (as between denoising steps)")
    ap.add_argument("--kv-heads", type=int, default=0,
                    help="grouped-query attention: K/V heads (a divisor of the query heads; "
                         "K/V are every G-th generated head); 0 = one per query head")
    ap.add_argument("--partition", default="response", choices=["response", "semantic", "key-response"],
                    help="partition ablation (Sec. 5.2): response-coupled (the method), semantic "
                         "(k-means on the raw keys and queries), key-response K/V groups with "
                         "semantic query groups")
    ap.add_argument("--probe-rule", default="stratified", choices=["stratified", "random", "uniform"],
                    help="probe-selection ablation (Table probe_estimator_ablation)")
    ap.add_argument("--routing", default="priority", choices=["priority", "top-p"],
                    help="routing rule: cost-aware greedy on the cell priorities (the default "
                         "reading) or per-group top-p with one p fitted to the budget")
    ap.add_argument("--ridge-only", action="store_true",
                    help="estimator ablation: ridge fit without the probe-residual subspace")
    ap.add_argument("--n-probes", type=int, default=-1,
                    help="probe rows per head (default: the workload's; 0 disables the repair)")
    ap.add_argument("--copy-probe", action="store_true",
                    help="run one plain fp32 copy (x * 1 over 256 MiB in, 256 MiB out) before the "
                         "timed region, so hardware counters of a known traffic can calibrate "
                         "those of the attention kernel")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: every SparsePR head is an independent call, and "
              "the library has no multi-GPU path (heads would shard across GPUs without any "
              "collective). Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2608_18484_amd import sparsepr as S
    S.lib()  # fail loudly if the HIP library is missing

    wl = W.CONFIGS[args.workload]
    t0 = time.perf_counter()
    q, k, v, host = generate(wl, torch)
    log(f"inputs {tuple(q.shape)} {q.dtype} generated in {time.perf_counter() - t0:.1f}s")

    p = params_for(S, wl, args.density)
    p.partition = {"response": 0, "semantic": 1, "key-response": 2}[args.partition]
    p.probe_rule = {"stratified": 0, "random": 1, "uniform": 2}[args.probe_rule]
    p.ridge_only = int(args.ridge_only)
    p.routing = {"priority": 0, "top-p": 1}[args.routing]
    if args.n_probes >= 0:
        p.n_probes = args.n_probes
    gqa = args.kv_heads > 0 and args.kv_heads != wl.heads
    default_cfg = (args.density == 0.25 and not gqa and not args.warm_start
                   and args.partition == "response" and args.probe_rule == "stratified"
                   and args.routing == "priority" and not args.ridge_only and args.n_probes < 0)
    if gqa:
        if wl.heads % args.kv_heads:
            print("--kv-heads must divide the query heads", file=sys.stderr)
            sys.exit(2)
        g = wl.heads // args.kv_heads
        k, v = k[:, ::g].contiguous(), v[:, ::g].contiguous()
    inputs = [(q, k, v)]
    if args.warm_start:
        p.warm_start, p.warm_iters = 1, 2
        gen = torch.Generator(device=q.device)
        gen.manual_seed(1234)

        def nudge(x):
            xf = x.float()
            noise = torch.randn(xf.shape, generator=gen, device=x.device, dtype=torch.float32)
            return (xf + 0.05 * xf.std() * noise).to(x.dtype)

        inputs.append(tuple(nudge(x) for x in (q, k, v)))
    op = S.SparsePR(S.shape_of(q, kv=k if gqa else None), p)
    out = torch.empty_like(q)
    stream = torch.cuda.current_stream()
    ncall = [0]

    def call():
        qi, ki, vi = inputs[ncall[0] % len(inputs)]
        ncall[0] += 1
        op.plan(qi, ki, stream)
        op.attend(qi, ki, vi, out, stream)

    for _ in range(args.warmup):
        call()
    torch.cuda.synchronize()
    log("warmup done")
    if args.copy_probe:
        src = torch.ones(64 << 20, dtype=torch.float32, device=q.device)
        dst = torch.empty_like(src)
        torch.mul(src, 1.0, out=dst)
        torch.cuda.synchronize()
        del src, dst
        log("copy probe: 268435456 bytes read, 268435456 bytes written")

    # timed region: K whole calls bracketed by synchronisation
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    ev0.record(stream)
    for _ in range(args.steps):
        call()
    ev1.record(stream)
    torch.cuda.synchronize()
    ms_per_call = ev0.elapsed_time(ev1) / args.steps
    st = op.stats(stream)
    log(f"{ms_per_call:.3f} ms per call, rho_exec {st['rho_exec']:.4f}")

    # per-phase device times with HIP events recorded by the library on the
    # same stream (a ring of events, no synchronisation inside the loop)
    op.set_profiling(True)
    for _ in range(args.steps):
        call()
    tm = op.timings(reset=True, stream=stream)
    op.set_profiling(False)
    n_calls = max(tm["attend_calls"], 1)
    nseg = tm["attn_launches"]
    attn_ms = tm["sparse_attn_ms"] / n_calls
    phases = {kk: round(tm[kk] / max(tm["plan_calls" if kk == "plan_ms" else "attend_calls"], 1), 4)
              for kk in ("plan_ms", "sparse_attn_ms", "probe_ms", "fit_ms", "correct_ms")}
    log(f"phases (ms/call): {phases}")

    d = wl.d
    exec_flops = 4.0 * d * st["exec_pairs"]
    tflops = exec_flops / (ms_per_call / 1e3) / 1e12
    # the dominant kernel: block-sparse attention over the routed pairs
    attn_flops = 4.0 * d * st["routed_pairs"]
    attn_tflops = attn_flops / (attn_ms / 1e3) / 1e12

    result = {
        "metric": "ms/attention call + effective TFLOP/s at 25% density; rel-L2 vs dense attn",
        "value": round(tflops, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_call, 4),
        "ms_per_call": round(ms_per_call, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if wl.dtype == "bf16" else "f32",
        "data": "synthetic (seeded random-Fourier-feature video tokens)",
        "config": {"workload": f"{wl.name}: {wl.grid[0]}x{wl.grid[1]}x{wl.grid[2]} grid, "
                               f"N={wl.n}, {wl.batch}x{wl.heads} heads, d={d}",
                   "n": wl.n, "heads": wl.batch * wl.heads, "d": d,
                   "target_exec_density": args.density, "kv_groups": wl.groups()[0],
                   "q_groups": wl.groups()[1], "probes": p.n_probes, "resid_rank": wl.resid_rank,
                   "kv_heads": wl.batch * (args.kv_heads if gqa else wl.heads),
                   "partition": args.partition, "probe_rule": args.probe_rule,
                   "routing": args.routing,
                   "estimator": "ridge only" if args.ridge_only else "ridge + probe-residual subspace",
                   "ridge": wl.ridge, "kmeans_iters": wl.kmeans_iters,
                   "kmeans_start": ("warm: 2 assignments from the previous call's centroids, "
                                    "inputs alternating with a 5%-noise copy")
                   if args.warm_start else "cold (strided rows)"},
        "rho_exec": round(st["rho_exec"], 6),
        "rho_route": round(st["rho_route"], 6),
        "exec_pairs": st["exec_pairs"],
        "kmeans_assignments": [st["kmeans_iters_kv"], st["kmeans_iters_q"]],
        "kmeans_exact_rescans": st["kmeans_rescans"],
        "phase_ms": phases,
        "roofline": {"bound": "mfma", "kernel": "k_attn_mfma<128, MODE_SPARSE>",
                     "achieved": round(attn_tflops, 2), "peak": BF16_PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(attn_tflops / BF16_PEAK_TFLOPS, 4),
                     "kernel_ms": round(attn_ms, 4),
                     # counters were taken on the default configuration only
                     "traffic": attn_traffic(wl.name) if default_cfg else None,
                     "unit_of_work": f"one call's sparse-attention launches ({nseg} key segments)"},
    }

    dense = None
    if not args.no_dense:
        ql, kl, vl = inputs[(ncall[0] - 1) % len(inputs)]  # the inputs of the last call
        dense = S.dense_attention(ql, kl, vl, stream=stream)
        # the same inputs through the library's dense attention (every key,
        # the block-sparse kernel's MFMA layout), timed over three calls for
        # the attention-level speedup of the whole SparsePR call
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        ev0.record(stream)
        for _ in range(3):
            S.dense_attention(ql, kl, vl, out=dense, stream=stream)
        ev1.record(stream)
        torch.cuda.synchronize()
        result["dense_ms"] = round(ev0.elapsed_time(ev1) / 3, 4)
        result["speedup_vs_dense"] = round(result["dense_ms"] / result["ms_per_call"], 3)
        log(f"dense attention {result['dense_ms']:.3f} ms per call; SparsePR call speedup "
            f"{result['speedup_vs_dense']:.2f}x")
        o = out.float()
        dn = dense.float()
        diff = (o - dn).reshape(-1, d)
        ref = dn.reshape(-1, d)
        rel = (diff.norm() / ref.norm()).item()
        row = diff.norm(dim=1) / ref.norm(dim=1).clamp_min(1e-30)
        result["rel_l2_vs_dense"] = round(rel, 6)
        result["row_err_mean"] = round(row.mean().item(), 6)
        result["row_err_p99"] = round(torch.quantile(row[:: max(1, row.numel() // 1000000)], 0.99).item(), 6)
        log(f"rel-L2 vs dense {rel:.5f}")
        # the same plan with the repair off: the hard-drop output of every row
        # (probe rows included), read back head by head from the workspace
        num = den = 0.0
        for bh in range(wl.batch * wl.heads):
            b, h = divmod(bh, wl.heads)
            osp = torch.from_numpy(op.export(bh, fields=["o_sparse"])["o_sparse"]).to(q.device)
            dh = dn[b, h]
            num += (osp - dh).double().pow(2).sum().item()
            den += dh.double().pow(2).sum().item()
        result["rel_l2_hard_drop"] = round((num / den) ** 0.5, 6)
        log(f"rel-L2 vs dense of the hard-drop output (repair off) {result['rel_l2_hard_drop']:.5f}")
        del o, dn, diff, ref, row

    if not args.no_cpu_baseline:
        log(f"CPU oracle on {args.cpu_heads} head(s) ...")
        result["cpu_baseline"] = cpu_baseline(wl, host, args.density, args.cpu_heads)
        log(f"CPU oracle: {result['cpu_baseline']['seconds']:.1f}s")
        if dense is not None and not args.warm_start and not gqa:
            result["dense_crosscheck"] = dense_crosscheck(wl, host, dense, out)
            log(f"dense cross-check: {result['dense_crosscheck']}")

    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
