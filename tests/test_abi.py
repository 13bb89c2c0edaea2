"""Host-side checks of the C ABI: the library loads, exports exactly what
include/sparsepr.h declares, and validates arguments before any HIP call."""
import ctypes
import os
import re
import subprocess

import pytest

from paper_2608_18484_amd import sparsepr as S

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sparsepr.h")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(sparsepr_[a-z_]+)\s*\(", src)))


def test_header_declares_the_binding_names():
    assert declared_functions() == sorted(S.EXPORTED)


def test_library_exports_every_declared_symbol():
    lib = S.lib()
    out = subprocess.check_output(["nm", "-D", "--defined-only", S.LIB_PATH], text=True)
    exported = {l.split()[-1] for l in out.splitlines() if " T " in l}
    for name in declared_functions():
        assert name in exported, name
        assert hasattr(lib, name)


def test_struct_layout_matches_c_compiler(tmp_path):
    # the binding's structs must have the C layout the header gives them
    structs = {"sparsepr_shape": S.Shape, "sparsepr_params": S.Params,
               "sparsepr_stats": S.Stats, "sparsepr_plan_host": S.PlanHost,
               "sparsepr_timings": S.Timings}
    lines = ['#include <stdio.h>', '#include <stddef.h>', f'#include "{HEADER}"', 'int main(void) {']
    for cname, cls in structs.items():
        lines.append(f'printf("{cname} %zu\\n", sizeof({cname}));')
        for fname, _ in cls._fields_:
            lines.append(f'printf("{cname}.{fname} %zu\\n", offsetof({cname}, {fname}));')
    lines.append("return 0; }")
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines))
    exe = tmp_path / "layout"
    subprocess.check_call(["gcc", "-o", str(exe), str(src)])
    got = dict(l.split() for l in subprocess.check_output([str(exe)], text=True).splitlines())
    for cname, cls in structs.items():
        assert int(got[cname]) == ctypes.sizeof(cls), cname
        for fname, _ in cls._fields_:
            assert int(got[f"{cname}.{fname}"]) == getattr(cls, fname).offset, (cname, fname)


def _ws(shape, params):
    n = ctypes.c_size_t(0)
    st = S.lib().sparsepr_workspace_size(ctypes.byref(shape), ctypes.byref(params), ctypes.byref(n))
    return st, n.value, S.lib().sparsepr_last_error().decode()


def tiny_shape(**kw):
    base = dict(batch=1, heads=1, n_q=1024, n_kv=1024, d=64, d_v=64, stride_b=65536,
                stride_h=65536, stride_n=64, dtype=S.F32)
    base.update(kw)
    return S.Shape(**base)


def test_defaults_follow_paper_table():
    p = S.default_params()
    assert (p.r_k, p.r_q, p.n_probes, p.resid_rank) == (48, 64, 64, 16)
    assert abs(p.ridge - 0.1) < 1e-7 and abs(p.target_exec_density - 0.22) < 1e-7
    assert abs(p.eps_q - 1e-6) < 1e-12


def test_workspace_size_ok_and_monotone():
    st, n1, _ = _ws(tiny_shape(), S.default_params(n_probes=32))
    assert st == 0 and n1 > 0
    st, n2, _ = _ws(tiny_shape(heads=4, stride_b=4 * 65536), S.default_params(n_probes=32))
    assert st == 0 and n2 > 3 * n1
    # grouped-query attention: plans per K/V head, attend outputs per query head
    st, n3, _ = _ws(tiny_shape(heads=4, stride_b=4 * 65536, heads_kv=2, kv_stride_b=2 * 65536,
                               kv_stride_h=65536), S.default_params(n_probes=32))
    assert st == 0 and n1 < n3 < n2


@pytest.mark.parametrize("shape_kw,param_kw,status,needle", [
    (dict(d=96, d_v=96, stride_n=96), {}, 2, "d must be 64 or 128"),
    (dict(d_v=128), {}, 2, "d must equal d_v"),
    (dict(n_kv=512), {}, 2, "self-attention"),
    (dict(batch=0), {}, 1, "batch"),
    (dict(dtype=7), {}, 1, "dtype"),
    (dict(stride_n=32), {}, 1, "stride"),
    ({}, dict(target_exec_density=0.0), 1, "target_exec_density"),
    ({}, dict(target_exec_density=1.5), 1, "target_exec_density"),
    ({}, dict(resid_rank=0), 1, "resid_rank"),
    ({}, dict(resid_rank=65), 1, "resid_rank"),
    ({}, dict(n_kv_groups=2000), 1, "group counts"),
    ({}, dict(n_probes=-1), 1, "n_probes"),
    ({}, dict(ridge=-1.0), 1, "ridge"),
    ({}, dict(n_dense_prefix=1024), 1, "n_dense_prefix"),
    ({}, dict(kmeans_iters=0), 1, "kmeans_iters"),
    ({}, dict(partition=3), 1, "partition"),
    ({}, dict(probe_rule=-1), 1, "probe_rule"),
    ({}, dict(ridge_only=2), 1, "ridge_only"),
    ({}, dict(routing=2), 1, "routing"),
    (dict(n_q=8192, n_kv=8192, stride_b=8192 * 64, stride_h=8192 * 64),
     dict(routing=1, n_kv_groups=5000), 2, "top-p"),
    (dict(n_q=4096, n_kv=4096, stride_b=4096 * 64, stride_h=4096 * 64), dict(probe_rule=1, n_probes=2000),
     2, "random probe rule"),
    (dict(heads=4, stride_b=4 * 65536, heads_kv=3), {}, 1, "heads_kv"),
    (dict(heads=4, stride_b=4 * 65536, heads_kv=-1), {}, 1, "heads_kv"),
    (dict(heads=4, stride_b=4 * 65536, heads_kv=2), {}, 1, "kv_stride"),
    (dict(heads=4, stride_b=4 * 65536, heads_kv=2, kv_stride_b=2 * 65536, kv_stride_h=65540), {}, 2,
     "multiples of 8"),
])
def test_validation_errors(shape_kw, param_kw, status, needle):
    st, _, msg = _ws(tiny_shape(**shape_kw), S.default_params(**param_kw))
    assert st == status and needle in msg


def test_null_arguments_rejected():
    lib = S.lib()
    assert lib.sparsepr_workspace_size(None, None, None) == 1
    assert lib.sparsepr_plan(None, None, None, None) == 1
    assert lib.sparsepr_attend(None, None, None, None, None, None) == 1
    assert lib.sparsepr_get_stats(None, None, None) == 1
    assert lib.sparsepr_plan_export(None, 0, None, None) == 1
    assert lib.sparsepr_plan_import(None, 0, None, None) == 1
    assert lib.sparsepr_set_profiling(None, 1) == 1
    assert lib.sparsepr_get_timings(None, None, 0, None) == 1
    lib.sparsepr_plan_destroy(None)
    sh = tiny_shape()
    p = S.default_params()
    h = ctypes.c_void_p()
    # NULL / misaligned workspace fail before touching the device
    assert lib.sparsepr_plan_create(ctypes.byref(sh), ctypes.byref(p), None, 0, ctypes.byref(h)) == 1
    assert lib.sparsepr_plan_create(ctypes.byref(sh), ctypes.byref(p), ctypes.c_void_p(16), 1 << 30,
                                    ctypes.byref(h)) == 1
    # too small a workspace
    assert lib.sparsepr_plan_create(ctypes.byref(sh), ctypes.byref(p), ctypes.c_void_p(1 << 20), 256,
                                    ctypes.byref(h)) == 3
    assert "needs" in lib.sparsepr_last_error().decode()


# --- the binding checks tensors against the plan's geometry before any launch

def _t(shape, dtype="float32", stride=None):
    import torch
    dt = getattr(torch, dtype)
    t = torch.zeros(shape, dtype=dt)
    if stride is not None:
        t = torch.empty_strided(shape, stride, dtype=dt)
    return t


def _plan_shape(**kw):
    base = dict(batch=1, heads=4, n_q=96, n_kv=96, d=64, d_v=64, stride_b=4 * 96 * 64,
                stride_h=96 * 64, stride_n=64, dtype=S.F32)
    base.update(kw)
    return S.Shape(**base)


def test_check_tensors_accepts_matching_tensors():
    sh = _plan_shape()
    x = _t((1, 4, 96, 64))
    S.check_tensors(sh, q=x, k=x, v=x, out=x.clone(), device_type="cpu")
    # grouped-query attention: K/V with their own head count and strides
    g = _plan_shape(heads_kv=2, kv_stride_b=2 * 96 * 64, kv_stride_h=96 * 64)
    kv = _t((1, 2, 96, 64))
    S.check_tensors(g, q=x, k=kv, v=kv, out=x, device_type="cpu")


@pytest.mark.parametrize("name,bad,needle", [
    ("q", dict(dtype="bfloat16"), "dtype"),
    ("out", dict(dtype="bfloat16"), "dtype"),
    ("k", dict(shape=(1, 3, 96, 64)), "shape"),
    ("v", dict(shape=(1, 4, 95, 64)), "shape"),
    ("out", dict(shape=(1, 4, 96, 32)), "shape"),
    ("q", dict(shape=(2, 4, 96, 64)), "shape"),
    ("v", dict(stride=(4 * 96 * 128, 96 * 128, 128, 1)), "strides"),
    ("out", dict(stride=(4 * 96 * 64, 64, 4 * 64, 1)), "strides"),
])
def test_check_tensors_rejects_mismatch(name, bad, needle):
    sh = _plan_shape()
    tens = {n: _t((1, 4, 96, 64)) for n in ("q", "k", "v", "out")}
    tens[name] = _t(bad.get("shape", (1, 4, 96, 64)), bad.get("dtype", "float32"), bad.get("stride"))
    with pytest.raises(ValueError, match=needle):
        S.check_tensors(sh, device_type="cpu", **tens)


def test_check_tensors_rejects_host_tensor_and_wrong_kv_heads():
    sh = _plan_shape()
    x = _t((1, 4, 96, 64))
    with pytest.raises(ValueError, match="expected a cuda tensor"):
        S.check_tensors(sh, q=x)
    g = _plan_shape(heads_kv=2, kv_stride_b=2 * 96 * 64, kv_stride_h=96 * 64)
    with pytest.raises(ValueError, match="shape"):
        S.check_tensors(g, q=x, k=x, device_type="cpu")
    with pytest.raises(ValueError, match="torch.Tensor"):
        S.check_tensors(sh, q=x.numpy(), device_type="cpu")


def test_op_methods_check_before_launch():
    # an op whose handle was never created: a launch would fail in the library,
    # so a ValueError proves the check runs first
    op = object.__new__(S.SparsePR)
    op.shape = _plan_shape()
    op.handle = ctypes.c_void_p()
    x = _t((1, 4, 96, 64))
    with pytest.raises(ValueError):
        op.plan(x, x)
    with pytest.raises(ValueError):
        op.attend(x, x, x, x)
    with pytest.raises(ValueError, match="expected a cuda tensor"):
        S.dense_attention(x, x, x, x)
