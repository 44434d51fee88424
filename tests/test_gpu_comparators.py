"""The comparators on the GPU against the oracle: the per-query bisection
baseline (float32, one thread per row) reaches the threshold of Eq. (1)
within the error its float32 sums allow, and DFTopK matches the oracle's
map, threshold, boundary pair and vector-Jacobian product."""
import math

import numpy as np
import pytest

import oracle.lapsum_oracle as O
import workloads as W
from test_gpu_parity import _np, _t, grad_rel

pytestmark = pytest.mark.gpu


def _bisect_budget_tol(r32, b, alpha, k):
    """|LapSum(b) - k| for the float32 baseline: a sequential float32 sum of
    n terms each within 2 ulp (|LapSum| <= k near the root: (n + 4) 2^-24 k),
    the float32 rounding of u = (r - mid)/t (2^-23 |u| relative on each term,
    at most 2^-20 k overall), and the float32 resolution of the midpoint
    (2 ulp of |b| + 1 times the slope sum f)."""
    t = -alpha
    r = np.asarray(r32, np.float64)
    F = float(np.sum(np.exp(-np.abs(r - b) / t))) / (2.0 * t)
    return (r.size + 4) * 2.0 ** -24 * k + 2.0 ** -20 * k + 2.0 ** -22 * (abs(b) + 1.0) * F


@pytest.mark.parametrize("batch,n,k,alpha", [(256, 4096, 256.0, -1.0), (3, 1000, 62.5, -0.05),
                                             (2, 7, 3.5, -2.0), (4, 1, 0.25, -0.5)])
def test_bisection_baseline_reaches_the_root(lib, batch, n, k, alpha):
    r = W.random_case(47, n, dist="normal", batch=batch)
    p, b = lib.lapsum_bisect_forward(_t(r), k, alpha, steps=60)
    p, b = _np(p), _np(b)
    pf, bf = lib.lapsum_forward(_t(r), k, alpha)
    pf = _np(pf)
    worst = 0.0
    for i in range(batch):
        tol = _bisect_budget_tol(r[i], float(b[i]), alpha, k)
        assert abs(O.lapsum(r[i], float(b[i]), -alpha) - k) <= tol, (i, b[i])
        # p is the Laplace CDF at the baseline's own b, in float32
        assert np.max(np.abs(p[i].astype(np.float64) - O.probs(r[i], float(b[i]), alpha))) <= 1e-6
        worst = max(worst, float(np.max(np.abs(p[i].astype(np.float64) - pf[i]))))
    # the fast path reproduces the baseline's mask (the paper: to 1.5e-5)
    assert worst <= 2e-5, worst


@pytest.mark.parametrize("n,k,dist,batch", [
    (10, 5, "normal", 1), (1000, 500, "normal", 2), (1000, 1, "levels16", 1),
    (1000, 999, "levels16", 1), (100_003, 50_001, "student2", 1), (3_000_000, 1_500_000, "normal", 1)])
def test_dftopk_matches_oracle(lib, n, k, dist, batch):
    alpha = -0.1
    r = W.random_case(48, n, dist=dist, batch=batch, ties=0.05 if dist == "normal" else 0.0)
    g = W.random_case(49, n, dist="normal", batch=batch)
    p, c, pair = lib.lapsum_dftopk_forward(_t(r), k, alpha)
    grad = _np(lib.lapsum_dftopk_backward(_t(g), p, pair, alpha))
    p, c, pair = _np(p), _np(c), _np(pair)
    for i in range(batch):
        po, co, (ik, ik1) = O.dftopk(r[i], k, alpha)
        assert float(c[i]) == co and (int(pair[i, 0]), int(pair[i, 1])) == (ik, ik1), i
        assert np.max(np.abs(p[i].astype(np.float64) - po)) <= 1e-6, i
        ref = O.dftopk_vjp(r[i], k, alpha, g[i])
        assert grad_rel(grad[i], ref) <= 1e-5, (i, grad_rel(grad[i], ref))


def test_dftopk_budget_drift_on_the_table_setting(lib):
    # Table budget's setting: Gaussian scores, k = n/16, alpha = -1.  DFTopK's
    # mass drifts to about 3.46 k; Fast LapSum's stays at k.
    n = 1_000_000
    r = np.random.default_rng([51, n]).standard_normal(n).astype(np.float32)
    k = n // 16
    p, _, _ = lib.lapsum_dftopk_forward(_t(r[None, :]), k, -1.0)
    got = abs(math.fsum(_np(p)[0].astype(np.float64)) - k) / k
    want = abs(math.fsum(O.dftopk(r, k, -1.0)[0]) - k) / k
    assert abs(got - want) <= 1e-5 and abs(got - 2.46) <= 0.025, (got, want)
    pf, _ = lib.lapsum_forward(_t(r[None, :]), float(k), -1.0)
    assert O.budget_error(_np(pf)[0], k) / k < 1e-5
