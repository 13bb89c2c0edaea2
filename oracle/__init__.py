"""SparsePR CPU oracle: ctypes wrapper over the plain C reference.

TEST INFRASTRUCTURE ONLY: imported by the tests, by the smoke check and by
the benchmark's CPU-baseline leg; the GPU library never imports, links or
runs it.  Every function works on one attention head given float32 numpy
arrays and returns numpy arrays.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "sparsepr_oracle.c")
_LIB_PATH = os.path.join(_HERE, "libsparsepr_oracle.so")
# AddressSanitizer + UndefinedBehaviorSanitizer build of the same source, used
# when SPARSEPR_ORACLE_SANITIZE=1 (the process must preload the gcc runtimes,
# see sanitize_env())
_SAN_PATH = os.path.join(_HERE, "libsparsepr_oracle_san.so")
_lib = None

# Portable x86-64-v3 code (the library travels to other hosts); no
# floating-point contraction so every float expression is evaluated as written.
CFLAGS = ["-O3", "-march=x86-64-v3", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
          "-shared", "-fPIC", "-std=c11", "-Wall"]


SAN_FLAGS = ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
             "-fno-sanitize-recover=undefined"]


def _sanitized() -> bool:
    return os.environ.get("SPARSEPR_ORACLE_SANITIZE", "") == "1"


def build(force: bool = True, sanitize: bool = False) -> str:
    """Compile the oracle with gcc into oracle/libsparsepr_oracle.so, or with
    sanitize=True into oracle/libsparsepr_oracle_san.so (ASan + UBSan)."""
    sanitize = sanitize or _sanitized()
    path = _SAN_PATH if sanitize else _LIB_PATH
    if force or not os.path.exists(path):
        tmp = path + ".tmp"
        flags = CFLAGS + (SAN_FLAGS if sanitize else [])
        subprocess.check_call(["gcc", *flags, "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, path)
    return path


def sanitize_env() -> dict:
    """Environment for a process that loads the sanitizer builds: the gcc
    ASan/UBSan runtimes preloaded (the interpreter itself is not
    instrumented), leak checking off (the interpreter's own allocations)."""
    rt = [subprocess.check_output(["gcc", f"-print-file-name={n}"], text=True).strip()
          for n in ("libasan.so", "libubsan.so")]
    env = dict(os.environ)
    env.update({"LD_PRELOAD": " ".join(rt), "ASAN_OPTIONS": "detect_leaks=0:abort_on_error=1",
                "UBSAN_OPTIONS": "print_stacktrace=1:halt_on_error=1",
                "SPARSEPR_ORACLE_SANITIZE": "1"})
    return env


def lib():
    global _lib
    if _lib is None:
        path = _SAN_PATH if _sanitized() else _LIB_PATH
        if not os.path.exists(path):
            build(sanitize=_sanitized())
        _lib = ctypes.CDLL(path)
    return _lib


def _p(a):
    return a.ctypes.data_as(ctypes.c_void_p) if a is not None else None


def _f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


def _i32(a):
    return np.ascontiguousarray(a, dtype=np.int32)


def _i64(a):
    return np.ascontiguousarray(a, dtype=np.int64)


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def num_threads() -> int:
    return int(lib().or_num_threads())


def dense_rows(q, k, v, rows=None):
    q, k, v = _f32(q), _f32(k), _f32(v)
    n, d = q.shape
    dv = v.shape[1]
    rows = _i64(np.arange(n) if rows is None else rows)
    out = np.zeros((len(rows), dv), np.float64)
    lib().or_dense_rows(_p(q), _p(k), _p(v), k.shape[0], d, dv, _p(rows), len(rows), _p(out))
    return out


def sparse_rows(q, k, v, labels_q, labels_kv, z, rows=None):
    q, k, v = _f32(q), _f32(k), _f32(v)
    n, d = q.shape
    dv = v.shape[1]
    z = np.ascontiguousarray(z, dtype=np.uint8)
    rows = _i64(np.arange(n) if rows is None else rows)
    out = np.zeros((len(rows), dv), np.float64)
    lib().or_sparse_rows(_p(q), _p(k), _p(v), k.shape[0], d, dv, _p(_i32(labels_q)),
                         _p(_i32(labels_kv)), z.shape[1], _p(z), _p(rows), len(rows), _p(out))
    return out


def key_metric(q, m_s):
    q = _f32(q)
    n, d = q.shape
    out = np.zeros((d, d), np.float64)
    lib().or_key_metric(_p(q), n, d, m_s, _p(out))
    return out


def key_metric_pooled(q, m_s):
    """M_K pooled over the query heads of q [G, n, d] (their mean)."""
    q = _f32(q)
    nh, n, d = q.shape
    out = np.zeros((d, d), np.float64)
    lib().or_key_metric_pooled(_p(q), nh, n, d, m_s, _p(out))
    return out


def project_pooled(x, f, eps=1e-6, rms=True):
    """Mean over the heads of x [G, n, d] of the (normalised) query coordinates."""
    x, f = _f32(x), _f64(f)
    nh, n, d = x.shape
    r = f.shape[1]
    phi = np.zeros((n, r), np.float32)
    lib().or_project_pooled(_p(x), nh, n, d, _p(f), r, int(rms), ctypes.c_double(eps), _p(phi))
    return phi


def splitmix64(x):
    lib().or_splitmix64.restype = ctypes.c_uint64
    return int(lib().or_splitmix64(ctypes.c_uint64(x)))


def probe_uniform(n, m):
    probes = np.zeros(max(m, 1), np.int32)
    w = np.zeros(max(m, 1), np.float64)
    k = lib().or_probe_uniform(n, m, _p(probes), _p(w))
    return probes[:k], w[:k]


def probe_random(n, m, seed):
    probes = np.zeros(max(m, 1), np.int32)
    w = np.zeros(max(m, 1), np.float64)
    k = lib().or_probe_random(n, m, ctypes.c_uint32(seed), _p(probes), _p(w))
    return probes[:k], w[:k]


def group_mean_pooled(x, labels, c):
    """Group means over the heads and members of x [G, n, d]."""
    x = _f32(x)
    nh, n, d = x.shape
    mean = np.zeros((c, d), np.float32)
    lib().or_group_mean_pooled(_p(x), nh, n, d, _p(_i32(labels)), c, _p(mean))
    return mean


def sym_eig(a):
    a = _f64(a)
    n = a.shape[0]
    ev = np.zeros(n, np.float64)
    u = np.zeros((n, n), np.float64)
    lib().or_sym_eig(_p(a), n, _p(ev), _p(u))
    return ev, u


def response_basis(m, r, tau=1e-6):
    m = _f64(m)
    d = m.shape[0]
    r = min(r, d)
    f = np.zeros((d, r), np.float64)
    ev = np.zeros(d, np.float64)
    lib().or_response_basis(_p(m), d, r, ctypes.c_double(tau), _p(f), _p(ev))
    return f, ev


def project(x, f, rms=False, eps=1e-6):
    x, f = _f32(x), _f64(f)
    n, d = x.shape
    r = f.shape[1]
    phi = np.zeros((n, r), np.float32)
    lib().or_project(_p(x), n, d, _p(f), r, int(rms), ctypes.c_double(eps), _p(phi))
    return phi


def kmeans(pts, c, iters, init=None):
    """Lloyd k-means; cold start from the strided points, or warm start from
    the centroids `init` (c x r) when given."""
    pts = _f32(pts)
    n, r = pts.shape
    labels = np.zeros(n, np.int32)
    cent = np.zeros((c, r), np.float32)
    counts = np.zeros(c, np.int32)
    if init is None:
        it = lib().or_kmeans(_p(pts), n, r, c, iters, _p(labels), _p(cent), _p(counts))
    else:
        init = _f32(init)
        assert init.shape == (c, r)
        it = lib().or_kmeans_from(_p(pts), n, r, c, iters, _p(init), _p(labels), _p(cent),
                                  _p(counts))
    return labels, cent, counts, it


def kmeans_assign(pts, cent, want_scores=False):
    pts, cent = _f32(pts), _f32(cent)
    n, r = pts.shape
    c = cent.shape[0]
    labels = np.zeros(n, np.int32)
    scores = np.zeros((n, c), np.float32) if want_scores else None
    lib().or_kmeans_assign(_p(pts), n, r, _p(cent), c, _p(labels), _p(scores))
    return (labels, scores) if want_scores else labels


def group_mean(x, labels, c):
    x = _f32(x)
    n, d = x.shape
    mean = np.zeros((c, d), np.float32)
    counts = np.zeros(c, np.int32)
    lib().or_group_mean(_p(x), n, d, _p(_i32(labels)), c, _p(mean), _p(counts))
    return mean, counts


def query_metric(kbar, counts):
    kbar = _f32(kbar)
    c, d = kbar.shape
    out = np.zeros((d, d), np.float64)
    lib().or_query_metric(_p(kbar), _p(_i32(counts)), c, d, _p(out))
    return out


def stable_perm(labels, c):
    labels = _i32(labels)
    n = len(labels)
    perm = np.zeros(n, np.int32)
    off = np.zeros(c + 1, np.int32)
    lib().or_stable_perm(_p(labels), n, c, _p(perm), _p(off))
    return perm, off


def route_priorities(qbar, nq, kbar, nk):
    qbar, kbar = _f32(qbar), _f32(kbar)
    cq, d = qbar.shape
    ck = kbar.shape[0]
    prio = np.zeros((cq, ck), np.float32)
    lib().or_route_priorities(_p(qbar), _p(_i32(nq)), cq, _p(kbar), _p(_i32(nk)), ck, d, _p(prio))
    return prio


def route_select(prio, nq, nk, budget):
    prio = _f32(prio)
    cq, ck = prio.shape
    z = np.zeros((cq, ck), np.uint8)
    out = np.zeros(4, np.int64)
    lib().or_route_select(_p(prio), _p(_i32(nq)), cq, _p(_i32(nk)), ck, ctypes.c_int64(int(budget)),
                          _p(z), _p(out))
    return z, {"routed_pairs": int(out[0]), "forced_pairs": int(out[1]),
               "routed_cells": int(out[2]), "forced_cells": int(out[3])}


def route_topp_keys(prio, nq, nk):
    """Keys of the per-group top-p walk: -(mass ranked before each cell)."""
    prio = _f32(prio)
    cq, ck = prio.shape
    keys = np.zeros((cq, ck), np.float32)
    lib().or_route_topp_keys(_p(prio), _p(_i32(nq)), cq, _p(_i32(nk)), ck, _p(keys))
    return keys


def probe_select(phi, labels, cent, m):
    phi, cent = _f32(phi), _f32(cent)
    n, r = phi.shape
    c = cent.shape[0]
    probes = np.zeros(max(m, 1), np.int32)
    w = np.zeros(max(m, 1), np.float64)
    np_ = lib().or_probe_select(_p(phi), n, r, _p(_i32(labels)), c, _p(cent), m, _p(probes), _p(w))
    return probes[:np_], w[:np_]


def fit(x, od, w, r, lam, eps=1e-6, ridge_only=False):
    x, od, w = _f64(x), _f64(od), _f64(w)
    m, dv = x.shape if x.ndim == 2 else (0, od.shape[-1])
    mu_x = np.zeros(dv)
    s_x = np.zeros(dv)
    mu_r = np.zeros(dv)
    b = np.zeros((dv, dv))
    psi = np.zeros((dv, max(r, 1)))
    g = np.zeros((dv, dv))
    rank = ctypes.c_int(0)
    st = lib().or_fit(_p(x), _p(od), _p(w), m, dv, r, int(ridge_only), ctypes.c_double(lam),
                      ctypes.c_double(eps),
                      _p(mu_x), _p(s_x), _p(mu_r), _p(b), _p(psi), _p(g), ctypes.byref(rank))
    return {"status": st, "mu_x": mu_x, "s_x": s_x, "mu_r": mu_r, "b": b,
            "psi": psi[:, :rank.value], "g": g, "rank": rank.value}


def correct_rows(x, ft):
    x = _f64(x)
    n, dv = x.shape
    out = np.zeros_like(x)
    lib().or_correct_rows(_p(x), n, dv, _p(ft["mu_x"]), _p(ft["s_x"]), _p(ft["mu_r"]),
                          _p(_f64(ft["g"])), _p(out))
    return out


def plan(q, k, *, n_text=0, n_sampled, r_k, r_q, c_k, c_q, iters, density, n_probes,
         partition=0, probe_rule=0, probe_seed=0, routing=0):
    """Whole Response-Coupled Partitioning + routing + probe choice for one
    K/V head.  q is [n, d], or [G, n, d] for the G query heads that share the
    K/V head under grouped-query attention (the plan pools them)."""
    q, k = _f32(q), _f32(k)
    nqh = 1 if q.ndim == 2 else q.shape[0]
    n, d = q.shape[-2:]
    nv = n - n_text
    rk, rq = min(r_k, d), min(r_q, d)
    if partition == 1:
        rk = d
    if partition != 0:
        rq = d
    cq_t, ck_t = c_q + (n_text > 0), c_k + (n_text > 0)
    out = {
        "labels_q": np.zeros(n, np.int32), "labels_kv": np.zeros(n, np.int32),
        "z": np.zeros((cq_t, ck_t), np.uint8),
        "probes": np.zeros(max(n_probes, 1), np.int32), "w": np.zeros(max(n_probes, 1)),
        "fk": np.zeros((d, rk)), "fq": np.zeros((d, rq)),
        "phik": np.zeros((nv, rk), np.float32), "phiq": np.zeros((nv, rq), np.float32),
        "kbar": np.zeros((c_k, d), np.float32), "qbar": np.zeros((c_q, d), np.float32),
        "cqphi": np.zeros((c_q, rq), np.float32), "prio": np.zeros((c_q, c_k), np.float32),
        "stats": np.zeros(7, np.int64),
    }
    lib().or_plan(_p(q), nqh, _p(k), n, d, n_text, n_sampled, r_k, r_q, c_k, c_q, iters,
                  ctypes.c_double(density), n_probes, int(partition), int(probe_rule),
                  ctypes.c_uint32(probe_seed), int(routing), _p(out["labels_q"]), _p(out["labels_kv"]),
                  _p(out["z"]), _p(out["probes"]), _p(out["w"]), _p(out["fk"]), _p(out["fq"]),
                  _p(out["phik"]), _p(out["phiq"]), _p(out["kbar"]), _p(out["qbar"]),
                  _p(out["cqphi"]), _p(out["prio"]), _p(out["stats"]))
    npr = int(out["stats"][4])
    out["probes"] = out["probes"][:npr]
    out["w"] = out["w"][:npr]
    s = out["stats"]
    out["rho_route"] = s[0] / float(n) / float(n)
    out["rho_exec"] = out["rho_route"] + npr / float(n)
    return out


def attend(q, k, v, labels_q, labels_kv, z, probes, w, *, n_text=0, r, lam, eps=1e-6,
           ridge_only=False):
    """Sparse attention + exact probes + fit + correction for one head (double)."""
    q, k, v = _f32(q), _f32(k), _f32(v)
    n, d = q.shape
    dv = v.shape[1]
    z = np.ascontiguousarray(z, dtype=np.uint8)
    probes = _i32(probes)
    w = _f64(w)
    m = len(probes)
    out = np.zeros((n, dv), np.float64)
    fo = np.zeros(3 * dv + dv * dv, np.float64)
    st = lib().or_attend(_p(q), _p(k), _p(v), n, d, dv, n_text, _p(_i32(labels_q)),
                         _p(_i32(labels_kv)), z.shape[0], z.shape[1], _p(z),
                         _p(probes) if m else None, _p(w) if m else None, m, r, int(ridge_only),
                         ctypes.c_double(lam), ctypes.c_double(eps), _p(out), _p(fo))
    fit_out = {"status": st, "mu_x": fo[:dv], "s_x": fo[dv:2 * dv], "mu_r": fo[2 * dv:3 * dv],
               "g": fo[3 * dv:].reshape(dv, dv)}
    return out, fit_out


def run(q, k, v, **params):
    """plan + attend for one head; returns (output, plan)."""
    pl = plan(q, k, n_text=params.get("n_text", 0), n_sampled=params["n_sampled"],
              r_k=params["r_k"], r_q=params["r_q"], c_k=params["c_k"], c_q=params["c_q"],
              iters=params["iters"], density=params["density"], n_probes=params["n_probes"],
              partition=params.get("partition", 0), probe_rule=params.get("probe_rule", 0),
              probe_seed=params.get("probe_seed", 0), routing=params.get("routing", 0))
    ridge_only = bool(params.get("ridge_only", False))
    dv = np.shape(v)[-1]
    out, ft = attend(q, k, v, pl["labels_q"], pl["labels_kv"], pl["z"], pl["probes"], pl["w"],
                     n_text=params.get("n_text", 0), r=dv if ridge_only else params["r"],
                     lam=params["lam"], ridge_only=ridge_only)
    pl["fit"] = ft
    return out, pl


# --------------------------------------------------------------------------
# Diagnostics of Sec. 3.1 (observations O1 and O3)
# --------------------------------------------------------------------------

def support_sets(q, k, rows, alpha):
    """|D_i(alpha)| for each listed row and the membership marks of D_i
    (bool, len(rows) x n_k): the smallest set of highest-weight keys whose
    dense attention mass reaches alpha."""
    q, k = _f32(q), _f32(k)
    n_k, d = k.shape
    rows = _i32(rows)
    counts = np.zeros(len(rows), np.int32)
    member = np.zeros((len(rows), n_k), np.uint8)
    lib().or_support_sets(_p(q), _p(k), n_k, d, _p(rows), len(rows), ctypes.c_double(alpha),
                          _p(counts), _p(member))
    return counts, member.astype(bool)


def pooled_support(member):
    """gamma: size of the union of the rows' supports over n_k."""
    member = np.asarray(member, bool)
    return float(np.count_nonzero(member.any(axis=0))) / member.shape[1]


def affine_fraction(osp, r):
    """Affine-explainable fraction ||P_X R||^2 / ||R||^2 with X = [1, O_sp],
    the affine-orthogonal energy and ||R||^2."""
    osp, r = _f64(osp), _f64(r)
    n, dv = osp.shape
    out = np.zeros(3)
    rank = lib().or_affine_fraction(_p(osp), _p(r), n, dv, _p(out))
    return {"fraction": float(out[0]), "orthogonal": float(out[1]), "energy": float(out[2]),
            "rank": int(rank)}
