"""Pins of the oracle's Sec. 3.1 diagnostics (observations O1 and O3) and the
diagnostics on a synthetic workload for the two partitions.

O1: tau_i(alpha) = |D_i(alpha)| / N_k with D_i(alpha) the smallest set of
highest-weight keys holding attention mass alpha, gamma = |union of D_i| / N_k
over a query group's rows.  O3 (eq. projection_decomposition): the share of
the hard-drop residual R explained by an affine function of the sparse output,
||P_X R||^2 / ||R||^2 with X = [1, O_sp], and the energy left outside.
"""
import numpy as np
import pytest

from paper_2608_18484_amd import workloads as W


def planted(n=1024, d=16, supports=((3, 17, 40, 200),), big=40.0):
    """Query row t attends (almost) only to the keys in supports[t]: those
    keys score big, every other key 0."""
    q = np.zeros((len(supports), d), np.float32)
    k = np.zeros((n, d), np.float32)
    for t, sup in enumerate(supports):
        q[t, t] = 1.0
        k[list(sup), t] = big * np.sqrt(d)
    return q, k


def test_support_uniform_closed_form(orc):
    # q = 0: every key has weight exactly 2^-10, so reaching alpha = 3/4 needs
    # exactly 768 keys, the lowest indices (ties to the lower index).
    n = 1024
    q = np.zeros((1, 8), np.float32)
    k = np.random.default_rng(0).standard_normal((n, 8)).astype(np.float32)
    counts, member = orc.support_sets(q, k, [0], 0.75)
    assert counts[0] == 768
    assert np.array_equal(np.flatnonzero(member[0]), np.arange(768))
    counts, _ = orc.support_sets(q, k, [0], 1.0)
    assert counts[0] == n


def test_support_planted_sets(orc):
    # A row whose mass sits on s planted keys (weight 1/s each, short by a
    # relative e^-40 n) needs ceil(alpha * s) of them for alpha away from the
    # multiples of 1/s, and they are planted ones.
    sup = (3, 17, 40, 200, 511, 1000, 5, 6, 7, 8)
    q, k = planted(supports=(sup,))
    for alpha, want in ((0.85, 9), (0.93, 10), (0.25, 3), (0.05, 1)):
        counts, member = orc.support_sets(q, k, [0], alpha)
        assert counts[0] == want, alpha
        assert set(np.flatnonzero(member[0])) <= set(sup)
    counts, member = orc.support_sets(q, k, [0], 0.999)
    assert set(np.flatnonzero(member[0])) == set(sup)


def test_pooled_support(orc):
    # gamma of one row is its tau; of a row repeated, still its tau; of rows
    # with disjoint supports, the sum of their taus; overlapping supports pool
    # to the size of the union.
    s1, s2, s3 = (1, 2, 3, 4), (10, 11, 12, 13, 14), (3, 4, 10, 50)
    q, k = planted(supports=(s1, s2, s3))
    counts, member = orc.support_sets(q, k, [0, 1, 2, 0], 0.999)
    n = k.shape[0]
    assert orc.pooled_support(member[:1]) == counts[0] / n
    assert orc.pooled_support(member[[0, 3]]) == counts[0] / n
    assert orc.pooled_support(member[:2]) == (counts[0] + counts[1]) / n
    assert orc.pooled_support(member[:3]) == len(set(s1) | set(s2) | set(s3)) / n


def test_affine_fraction_special_cases(orc):
    rng = np.random.default_rng(3)
    n, dv = 400, 12
    osp = rng.standard_normal((n, dv))
    x = np.hstack([np.ones((n, 1)), osp])
    # exactly affine: all explained
    r = x @ rng.standard_normal((dv + 1, dv))
    a = orc.affine_fraction(osp, r)
    assert abs(a["fraction"] - 1.0) < 1e-9 and a["orthogonal"] < 1e-8 * a["energy"]
    # orthogonal to the feature space: nothing explained
    z = rng.standard_normal((n, dv))
    z -= x @ np.linalg.lstsq(x, z, rcond=None)[0]
    a = orc.affine_fraction(osp, z)
    assert a["fraction"] < 1e-9 and abs(a["orthogonal"] - a["energy"]) < 1e-9 * a["energy"]
    # general case against numpy's least squares (a library routine the
    # oracle does not use)
    r = rng.standard_normal((n, dv)) + 0.5 * (x @ rng.standard_normal((dv + 1, dv)))
    res = r - x @ np.linalg.lstsq(x, r, rcond=None)[0]
    want = 1.0 - np.sum(res ** 2) / np.sum(r ** 2)
    a = orc.affine_fraction(osp, r)
    assert abs(a["fraction"] - want) < 1e-9
    assert abs(a["orthogonal"] - np.sum(res ** 2)) < 1e-8 * np.sum(r ** 2)


def test_affine_fraction_depends_only_on_the_feature_space(orc):
    # X = [1, O_sp] spans the same space after O_sp -> O_sp T + 1 b^T (T
    # invertible), so the fraction is unchanged; a rank-deficient O_sp (a
    # repeated column) is handled; scaling R does not change the fraction.
    rng = np.random.default_rng(4)
    n, dv = 300, 8
    osp = rng.standard_normal((n, dv))
    r = rng.standard_normal((n, dv)) + osp @ rng.standard_normal((dv, dv))
    base = orc.affine_fraction(osp, r)["fraction"]
    t = rng.standard_normal((dv, dv)) + 3 * np.eye(dv)
    moved = osp @ t + rng.standard_normal(dv)
    assert abs(orc.affine_fraction(moved, r)["fraction"] - base) < 1e-8
    assert abs(orc.affine_fraction(osp, 7.5 * r)["fraction"] - base) < 1e-12
    dup = osp.copy()
    dup[:, 1] = dup[:, 0]
    a = orc.affine_fraction(dup, r)
    assert a["rank"] == dv
    x = np.hstack([np.ones((n, 1)), dup])
    res = r - x @ np.linalg.lstsq(x, r, rcond=None)[0]
    assert abs(a["fraction"] - (1.0 - np.sum(res ** 2) / np.sum(r ** 2))) < 1e-8


def diagnostics(orc, wl, partition, alpha=0.9, n_groups=8, m=16):
    """tau / gamma over the first rows of a few query groups and the O3
    decomposition of the hard-drop residual, for one head under a partition."""
    q, k, v, _ = W.make_inputs(wl)
    q, k, v = q[0, 0], k[0, 0], v[0, 0]
    ck, cq = wl.groups()
    pl = orc.plan(q, k, n_sampled=wl.n_sampled, r_k=48, r_q=64, c_k=ck, c_q=cq,
                  iters=wl.kmeans_iters, density=wl.density, n_probes=0, partition=partition)
    osp = orc.sparse_rows(q, k, v, pl["labels_q"], pl["labels_kv"], pl["z"])
    dense = orc.dense_rows(q, k, v)
    aff = orc.affine_fraction(osp, dense - osp)
    taus, gammas = [], []
    for a in range(0, cq, max(1, cq // n_groups))[:n_groups]:
        rows = np.flatnonzero(pl["labels_q"] == a)[:m]
        if len(rows) == 0:
            continue
        counts, member = orc.support_sets(q, k, rows, alpha)
        taus.extend(counts / k.shape[0])
        gammas.append(orc.pooled_support(member))
    return dict(tau=float(np.median(taus)), gamma=float(np.median(gammas)), **aff,
                rho=pl["rho_route"])


def test_diagnostics_on_the_tiny_workload(orc):
    # Both partitions at the same routing rule and density: the invariants of
    # the diagnostics (pooled support at least the row support, a fraction in
    # [0, 1], the energies adding up).  The values are reported, not pinned.
    wl = W.CONFIGS["tiny"]
    for partition in (0, 1):
        dg = diagnostics(orc, wl, partition)
        assert dg["gamma"] >= dg["tau"] > 0
        assert 0.0 <= dg["fraction"] <= 1.0
        assert abs(dg["orthogonal"] - (1 - dg["fraction"]) * dg["energy"]) < 1e-9 * dg["energy"]
        print(f"partition {partition}: tau {dg['tau']:.4f} gamma {dg['gamma']:.4f} "
              f"affine fraction {dg['fraction']:.4f} orthogonal {dg['orthogonal']:.4e}")
