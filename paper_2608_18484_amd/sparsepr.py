"""Thin ctypes binding of the SparsePR C ABI (include/sparsepr.h).

Argument marshalling only: every step of the operator runs in the HIP
library.  torch supplies device memory (inputs, outputs, the workspace) and
the stream.  Loading fails loudly when the library has not been built.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
# SPARSEPR_LIB selects another build of the same library (the host-side
# sanitizer build of build.py --sanitize); the default is the in-tree build
LIB_PATH = os.environ.get("SPARSEPR_LIB") or os.path.join(HERE, "libsparsepr.so")

F32, BF16 = 0, 1
FLAG_NONFINITE_INPUT, FLAG_FIT_NOT_PD, FLAG_BUDGET_BELOW_FORCED, FLAG_EIG_JACOBI = 1, 2, 4, 8
STATUS = {0: "OK", 1: "INVALID_ARGUMENT", 2: "UNSUPPORTED", 3: "WORKSPACE_TOO_SMALL", 4: "HIP",
          5: "NUMERICAL"}


class Shape(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("heads", ctypes.c_int32), ("n_q", ctypes.c_int32),
                ("n_kv", ctypes.c_int32), ("d", ctypes.c_int32), ("d_v", ctypes.c_int32),
                ("stride_b", ctypes.c_int64), ("stride_h", ctypes.c_int64),
                ("stride_n", ctypes.c_int64), ("dtype", ctypes.c_int32),
                ("heads_kv", ctypes.c_int32), ("kv_stride_b", ctypes.c_int64),
                ("kv_stride_h", ctypes.c_int64)]


class Params(ctypes.Structure):
    _fields_ = [("n_sampled_queries", ctypes.c_int32), ("r_k", ctypes.c_int32),
                ("r_q", ctypes.c_int32), ("n_kv_groups", ctypes.c_int32),
                ("n_q_groups", ctypes.c_int32), ("kmeans_iters", ctypes.c_int32),
                ("target_exec_density", ctypes.c_float), ("n_probes", ctypes.c_int32),
                ("resid_rank", ctypes.c_int32), ("ridge", ctypes.c_float),
                ("eps_q", ctypes.c_float), ("eps_x", ctypes.c_float),
                ("n_dense_prefix", ctypes.c_int32), ("warm_start", ctypes.c_int32),
                ("warm_iters", ctypes.c_int32), ("partition", ctypes.c_int32),
                ("probe_rule", ctypes.c_int32), ("probe_seed", ctypes.c_uint32),
                ("ridge_only", ctypes.c_int32), ("routing", ctypes.c_int32)]


class Stats(ctypes.Structure):
    _fields_ = [("rho_route", ctypes.c_double), ("rho_exec", ctypes.c_double),
                ("routed_pairs", ctypes.c_int64), ("exec_pairs", ctypes.c_int64),
                ("forced_pairs", ctypes.c_int64), ("routed_cells", ctypes.c_int32),
                ("forced_cells", ctypes.c_int32), ("nonempty_q_groups", ctypes.c_int32),
                ("nonempty_kv_groups", ctypes.c_int32), ("n_probes", ctypes.c_int32),
                ("kmeans_iters_kv", ctypes.c_int32), ("kmeans_iters_q", ctypes.c_int32),
                ("status_flags", ctypes.c_int32), ("kmeans_rescans", ctypes.c_int64)]


class Timings(ctypes.Structure):
    _fields_ = [("plan_ms", ctypes.c_double), ("sparse_attn_ms", ctypes.c_double),
                ("probe_ms", ctypes.c_double), ("fit_ms", ctypes.c_double),
                ("correct_ms", ctypes.c_double), ("plan_calls", ctypes.c_int32),
                ("attend_calls", ctypes.c_int32), ("attn_launches", ctypes.c_int32)]


_P = ctypes.c_void_p
HOST_FIELDS = [
    ("labels_q", "i4"), ("labels_kv", "i4"), ("routes", "u1"), ("probes", "i4"),
    ("n_probes", None),
    ("probe_weights", "f4"), ("perm_q", "i4"), ("off_q", "i4"), ("perm_kv", "i4"),
    ("off_kv", "i4"), ("m_k", "f4"), ("m_q", "f4"), ("f_k", "f4"), ("f_q", "f4"),
    ("phi_k", "f4"), ("phi_q", "f4"), ("cent_k", "f4"), ("cent_q", "f4"), ("kbar", "f4"),
    ("qbar", "f4"), ("route_prio", "f4"), ("o_sparse", "f4"), ("o_dense_probes", "f4"),
    ("fit_mu_x", "f4"), ("fit_s_x", "f4"), ("fit_mu_r", "f4"), ("fit_bpsi", "f4"),
    ("fit_psi", "f4"), ("fit_rank", None), ("route_key", "f4"),
]


class PlanHost(ctypes.Structure):
    _fields_ = [(name, ctypes.c_int32 if kind is None else _P) for name, kind in HOST_FIELDS]


EXPORTED = ["sparsepr_params_default", "sparsepr_workspace_size", "sparsepr_plan_create",
            "sparsepr_plan", "sparsepr_attend", "sparsepr_dense_workspace_size",
            "sparsepr_dense_attend", "sparsepr_get_stats", "sparsepr_plan_export",
            "sparsepr_plan_import", "sparsepr_set_profiling", "sparsepr_get_timings",
            "sparsepr_plan_destroy", "sparsepr_last_error", "sparsepr_plan_create_static"]

_lib = None


def lib():
    """Load libsparsepr.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"SparsePR HIP library not built: {LIB_PATH} is missing "
                               "(run __graft_entry__.build() or paper_2608_18484_amd/build.py)")
        L = ctypes.CDLL(LIB_PATH)
        L.sparsepr_last_error.restype = ctypes.c_char_p
        for name in EXPORTED:
            if name not in ("sparsepr_last_error", "sparsepr_params_default", "sparsepr_plan_destroy"):
                getattr(L, name).restype = ctypes.c_int
        _lib = L
    return _lib


class SparsePRError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status


def _check(st):
    if st != 0:
        raise SparsePRError(st, lib().sparsepr_last_error().decode())


PARTITION_RESPONSE, PARTITION_SEMANTIC, PARTITION_KEY_RESPONSE = 0, 1, 2
PROBES_STRATIFIED, PROBES_RANDOM, PROBES_UNIFORM = 0, 1, 2
ROUTING_PRIORITY, ROUTING_TOP_P = 0, 1


def default_params(**kw) -> Params:
    p = Params()
    lib().sparsepr_params_default(ctypes.byref(p))
    for k, v in kw.items():
        setattr(p, k, v)
    return p


def shape_of(t, dtype=None, kv=None) -> Shape:
    """Shape struct for a [B, H, N, d] torch tensor (last dim contiguous).
    `kv`: the [B, H_kv, N, d] K tensor (V must share its strides) for
    grouped-query attention, where H_kv divides H."""
    import torch
    b, h, n, d = t.shape
    sb, sh, sn, sd = t.stride()
    if sd != 1:
        raise ValueError("last dimension must be contiguous")
    dt = dtype if dtype is not None else (BF16 if t.dtype == torch.bfloat16 else F32)
    hkv, ksb, ksh = 0, 0, 0
    if kv is not None:
        bk, hkv, nk, dk = kv.shape
        ksb, ksh, ksn, ksd = kv.stride()
        if (bk, nk, dk) != (b, n, d) or ksn != sn or ksd != 1:
            raise ValueError("K/V must be [B, H_kv, N, d] with Q's row stride")
    return Shape(b, h, n, n, d, d, sb, sh, sn, dt, hkv, ksb, ksh)


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr())


def check_tensors(shape: Shape, q=None, k=None, v=None, out=None, device_type="cuda"):
    """Check tensors against the geometry a plan was created with, before any
    launch: the C side sees only pointers, so a tensor with another dtype,
    fewer heads or rows, or other strides would make the kernels read or write
    past its end.  Q and the output are [batch, heads, n, d] with the shape's
    strides; K and V are [batch, heads_kv, n, d] with the K/V strides (the Q
    strides when heads_kv is 0).  Raises ValueError on any mismatch."""
    import torch
    want_dtype = torch.bfloat16 if shape.dtype == BF16 else torch.float32
    hkv = shape.heads_kv or shape.heads
    kvsb = shape.kv_stride_b or shape.stride_b
    kvsh = shape.kv_stride_h or shape.stride_h
    geo = {
        "q": ((shape.batch, shape.heads, shape.n_q, shape.d),
              (shape.stride_b, shape.stride_h, shape.stride_n, 1)),
        "out": ((shape.batch, shape.heads, shape.n_q, shape.d_v),
                (shape.stride_b, shape.stride_h, shape.stride_n, 1)),
        "k": ((shape.batch, hkv, shape.n_kv, shape.d), (kvsb, kvsh, shape.stride_n, 1)),
        "v": ((shape.batch, hkv, shape.n_kv, shape.d_v), (kvsb, kvsh, shape.stride_n, 1)),
    }
    device = None
    for name, t in (("q", q), ("k", k), ("v", v), ("out", out)):
        if t is None:
            continue
        if not isinstance(t, torch.Tensor):
            raise ValueError(f"{name}: expected a torch.Tensor, got {type(t).__name__}")
        if t.device.type != device_type:
            raise ValueError(f"{name}: tensor on {t.device}, expected a {device_type} tensor")
        if device is None:
            device = t.device
        elif t.device != device:
            raise ValueError(f"{name}: tensor on {t.device}, the others on {device}")
        if t.dtype != want_dtype:
            raise ValueError(f"{name}: dtype {t.dtype}, the plan was made for {want_dtype}")
        dims, strides = geo[name]
        if tuple(t.shape) != dims:
            raise ValueError(f"{name}: shape {tuple(t.shape)}, the plan was made for {dims}")
        # a dimension of extent 1 is never stepped over, so its stride is free
        for ax, (got, exp) in enumerate(zip(t.stride(), strides)):
            if dims[ax] > 1 and got != exp:
                raise ValueError(f"{name}: strides {tuple(t.stride())}, the plan was made for "
                                 f"{strides}")


def _stream(stream):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


class SparsePR:
    """One SparsePR operator instance bound to a shape, parameters and a workspace."""

    def __init__(self, shape: Shape, params: Params, device="cuda", static=False):
        """static=True binds the plan to the library's static scratch array of
        the current device (sparsepr_plan_create_static: nothing is
        allocated; one such plan per device at a time, small shapes only)."""
        import torch
        self.shape, self.params = shape, params
        nbytes = ctypes.c_size_t(0)
        _check(lib().sparsepr_workspace_size(ctypes.byref(shape), ctypes.byref(params),
                                             ctypes.byref(nbytes)))
        self.workspace_bytes = nbytes.value
        self.handle = ctypes.c_void_p()
        if static:
            self.workspace = None
            _check(lib().sparsepr_plan_create_static(ctypes.byref(shape), ctypes.byref(params),
                                                     ctypes.byref(self.handle)))
        else:
            self.workspace = torch.empty(max(nbytes.value, 256), dtype=torch.uint8, device=device)
            _check(lib().sparsepr_plan_create(ctypes.byref(shape), ctypes.byref(params),
                                              _ptr(self.workspace),
                                              ctypes.c_size_t(self.workspace.numel()),
                                              ctypes.byref(self.handle)))
        n = shape.n_q
        ntext = params.n_dense_prefix
        nv = n - ntext
        self.ck = params.n_kv_groups or -(-nv // 64)
        self.cq = params.n_q_groups or -(-nv // 64)
        self.ck_t = self.ck + (ntext > 0)
        self.cq_t = self.cq + (ntext > 0)
        self.m = min(params.n_probes, nv)

    def close(self):
        """Destroy the plan handle now (a static plan releases its device's array)."""
        h = getattr(self, "handle", None)
        if h is not None and h.value and _lib is not None:
            _lib.sparsepr_plan_destroy(h)
        self.handle = None

    def __del__(self):
        self.close()

    def plan(self, q, k, stream=None):
        check_tensors(self.shape, q=q, k=k)
        _check(lib().sparsepr_plan(self.handle, _ptr(q), _ptr(k), _stream(stream)))

    def attend(self, q, k, v, out, stream=None):
        check_tensors(self.shape, q=q, k=k, v=v, out=out)
        _check(lib().sparsepr_attend(self.handle, _ptr(q), _ptr(k), _ptr(v), _ptr(out),
                                     _stream(stream)))

    def __call__(self, q, k, v, out=None, stream=None):
        import torch
        if out is None:
            out = torch.empty_like(q)
        self.plan(q, k, stream)
        self.attend(q, k, v, out, stream)
        return out

    def stats(self, stream=None) -> dict:
        s = Stats()
        _check(lib().sparsepr_get_stats(self.handle, ctypes.byref(s), _stream(stream)))
        return {name: getattr(s, name) for name, _ in Stats._fields_}

    def set_profiling(self, enable=True):
        _check(lib().sparsepr_set_profiling(self.handle, ctypes.c_int32(int(enable))))

    def timings(self, reset=True, stream=None) -> dict:
        t = Timings()
        _check(lib().sparsepr_get_timings(self.handle, ctypes.byref(t), ctypes.c_int32(int(reset)),
                                          _stream(stream)))
        return {name: getattr(t, name) for name, _ in Timings._fields_}

    def _sizes(self):
        sh, p = self.shape, self.params
        n, d, dv = sh.n_q, sh.d, sh.d_v
        nv = n - p.n_dense_prefix
        rk, rq = min(p.r_k, d), min(p.r_q, d)
        if p.partition == PARTITION_SEMANTIC:
            rk = d
        if p.partition != PARTITION_RESPONSE:
            rq = d
        r = dv if p.ridge_only else p.resid_rank
        m = max(self.m, 1)
        return {
            "labels_q": n, "labels_kv": n, "routes": self.cq_t * self.ck_t, "probes": m,
            "probe_weights": m, "perm_q": n, "off_q": self.cq_t + 1, "perm_kv": n,
            "off_kv": self.ck_t + 1, "m_k": d * d, "m_q": d * d, "f_k": d * rk, "f_q": d * rq,
            "phi_k": nv * rk, "phi_q": nv * rq, "cent_k": self.ck * rk, "cent_q": self.cq * rq,
            "kbar": self.ck * d, "qbar": self.cq * d, "route_prio": self.cq * self.ck,
            "route_key": self.cq * self.ck, "o_sparse": n * dv, "o_dense_probes": m * dv,
            "fit_mu_x": dv, "fit_s_x": dv,
            "fit_mu_r": dv, "fit_bpsi": dv * r, "fit_psi": dv * r,
        }

    def export(self, bh: int = 0, fields=None, stream=None) -> dict:
        """Copy the plan used by query head bh (and that head's attend outputs)
        to numpy arrays."""
        sizes = self._sizes()
        want = [name for name, kind in HOST_FIELDS if kind is not None and
                (fields is None or name in fields)]
        bufs = {}
        ph = PlanHost()
        for name, kind in HOST_FIELDS:
            if kind is None or name not in want:
                continue
            arr = np.zeros(sizes[name], dtype=np.dtype(kind))
            bufs[name] = arr
            setattr(ph, name, arr.ctypes.data_as(ctypes.c_void_p))
        _check(lib().sparsepr_plan_export(self.handle, ctypes.c_int32(bh), ctypes.byref(ph),
                                          _stream(stream)))
        sh, p = self.shape, self.params
        d, dv = sh.d, sh.d_v
        r = dv if p.ridge_only else p.resid_rank
        rk, rq = min(p.r_k, d), min(p.r_q, d)
        if p.partition == PARTITION_SEMANTIC:
            rk = d
        if p.partition != PARTITION_RESPONSE:
            rq = d
        npr = ph.n_probes
        shapes = {"routes": (self.cq_t, self.ck_t), "m_k": (d, d), "m_q": (d, d),
                  "f_k": (d, rk), "f_q": (d, rq), "phi_k": (-1, rk), "phi_q": (-1, rq),
                  "cent_k": (self.ck, rk), "cent_q": (self.cq, rq), "kbar": (self.ck, d),
                  "qbar": (self.cq, d), "route_prio": (self.cq, self.ck),
                  "route_key": (self.cq, self.ck), "o_sparse": (-1, dv),
                  "o_dense_probes": (-1, dv), "fit_bpsi": (dv, r), "fit_psi": (dv, r)}
        out = {}
        for name, arr in bufs.items():
            if name in ("probes", "probe_weights"):
                arr = arr[:npr]
            if name == "o_dense_probes":
                arr = arr[:npr * dv]
            out[name] = arr.reshape(shapes[name]) if name in shapes else arr
        out["n_probes"] = npr
        out["fit_rank"] = ph.fit_rank
        return out

    def import_plan(self, bh: int, labels_q, labels_kv, routes, probes, stream=None):
        """Replace the plan used by query head bh (shared by its K/V head's
        group) by host arrays (labels, route matrix, probes)."""
        lq = np.ascontiguousarray(labels_q, np.int32)
        lk = np.ascontiguousarray(labels_kv, np.int32)
        z = np.ascontiguousarray(routes, np.uint8)
        pr = np.ascontiguousarray(probes, np.int32)
        ph = PlanHost()
        ph.labels_q = lq.ctypes.data_as(ctypes.c_void_p)
        ph.labels_kv = lk.ctypes.data_as(ctypes.c_void_p)
        ph.routes = z.ctypes.data_as(ctypes.c_void_p)
        ph.probes = pr.ctypes.data_as(ctypes.c_void_p) if len(pr) else None
        ph.n_probes = len(pr)
        _check(lib().sparsepr_plan_import(self.handle, ctypes.c_int32(bh), ctypes.byref(ph),
                                          _stream(stream)))


def dense_attention(q, k, v, out=None, stream=None):
    """Dense attention (Sec. 3) for every query head on the probe kernels
    (K and V may have fewer heads: grouped-query attention)."""
    import torch
    if out is None:
        out = torch.empty_like(q)
    sh = shape_of(q, kv=k if k.shape[1] != q.shape[1] else None)
    check_tensors(sh, q=q, k=k, v=v, out=out)
    _check(lib().sparsepr_dense_attend(ctypes.byref(sh), _ptr(q), _ptr(k), _ptr(v), _ptr(out),
                                       None, ctypes.c_size_t(0), _stream(stream)))
    return out
