"""The allocation-free entry point (sparsepr_plan_create_static) against the
workspace entry point (sparsepr_plan_create), through the C ABI: identical
plans (labels, routes, probes bit-exact) and outputs, on two calls in a row,
the second with a smaller input; shapes beyond the static array are refused."""
import ctypes

import numpy as np
import pytest

from paper_2608_18484_amd import workloads as W
from tests._common import medium, params_for, rel_l2, to_device

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _call(S, wl, inputs, static):
    tq, tk, tv = inputs
    p = params_for(wl)
    op = S.SparsePR(S.shape_of(tq), p, static=static)
    assert (op.workspace is None) == static
    out = torch.empty_like(tq)
    op.plan(tq, tk)
    op.attend(tq, tk, tv, out)
    torch.cuda.synchronize()
    ex = [op.export(bh, fields=["labels_q", "labels_kv", "routes", "probes"])
          for bh in range(wl.batch * wl.heads)]
    st = op.stats()
    op.close()
    return out.float().cpu().numpy(), ex, st


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_static_plan_matches_workspace_plan(dtype):
    from paper_2608_18484_amd import sparsepr as S
    d = 128 if dtype == "bf16" else 64
    # two calls in a row on the static array, the second smaller
    for grid, heads in (((4, 24, 32), 3), ((2, 16, 32), 1)):
        wl = medium(grid=grid, heads=heads, dtype=dtype, d=d)
        print(f"\n[no-alloc] {dtype} grid {grid} heads {heads}", flush=True)
        q, k, v, _ = W.make_inputs(wl)
        inputs = to_device(q, k, v, wl.dtype)
        ref, ex_ref, st_ref = _call(S, wl, inputs, static=False)
        got, ex_got, st_got = _call(S, wl, inputs, static=True)
        for a, b in zip(ex_ref, ex_got):
            for key in ("labels_q", "labels_kv", "routes", "probes"):
                assert np.array_equal(a[key], b[key]), key
        assert st_ref["exec_pairs"] == st_got["exec_pairs"]
        assert st_got["status_flags"] == st_ref["status_flags"]
        assert rel_l2(got, ref) <= (2e-2 if dtype == "bf16" else 1e-5)
        assert np.array_equal(got, ref)  # same kernels, same plan: bit-identical


def test_static_plan_limits():
    from paper_2608_18484_amd import sparsepr as S
    wl = medium(grid=(2, 16, 32), heads=1)
    q, k, v, _ = W.make_inputs(wl)
    tq, tk, tv = to_device(q, k, v, wl.dtype)
    p = params_for(wl)
    op = S.SparsePR(S.shape_of(tq), p, static=True)
    # one plan per device holds the array
    with pytest.raises(S.SparsePRError, match="alive"):
        S.SparsePR(S.shape_of(tq), p, static=True)
    op.close()
    op2 = S.SparsePR(S.shape_of(tq), p, static=True)
    op2.close()
    # a shape whose workspace exceeds the array
    big = S.Shape(1, 24, 17160, 17160, 128, 128, 24 * 17160 * 128, 17160 * 128, 128, S.BF16, 0, 0, 0)
    pb = S.default_params(n_kv_groups=269, n_q_groups=269, n_probes=128)
    h = ctypes.c_void_p()
    st = S.lib().sparsepr_plan_create_static(ctypes.byref(big), ctypes.byref(pb), ctypes.byref(h))
    assert st == 3
    assert "static scratch array" in S.lib().sparsepr_last_error().decode()
