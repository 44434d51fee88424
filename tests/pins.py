"""Pin checks for the float64 oracle.

Each check ties an oracle routine to something the paper or the mathematics
fixes independently of the oracle's own code: a closed form, an invariant,
brute force at high precision, finite differences, or a theorem's
probability.  They are plain functions (raising AssertionError) so that the
planted-mistake tests can run them against deliberately broken copies of the
oracle.
"""
from __future__ import annotations

import math
from decimal import Decimal, getcontext

import numpy as np

import oracle.lapsum_oracle as O
import workloads as W


def _rows(seed_count=40):
    rg = np.random.default_rng(12345)
    for seed in range(seed_count):
        for dist in ("normal", "levels16", "cauchy", "clusters3", "laplace_abs"):
            n = int(rg.integers(2, 200))
            x = W.random_case(seed, n, dist=dist, ties=0.15)[0]
            k = float(rg.uniform(0.05, n - 0.05))
            a = -float(rg.choice([1e-3, 0.02, 0.3, 1.0, 7.0]))
            yield x, k, a


def check_bisect_matches_scan(seed_count=40):
    """Brute force (bisection on the plain sum) vs the sort-and-scan closed form."""
    for x, k, a in _rows(seed_count):
        b1 = O.solve_bisect(x, k, a)
        b2 = O.solve_sorted_scan(x, k, a)
        assert abs(b1 - b2) <= 1e-9 * -a + 1e-12 * abs(b1), (k, a, b1, b2)


def check_n1_closed_form():
    """n = 1: sigma((r - b)/t) = k gives b = r - t ln(2k) (k <= 1/2) and
    b = r + t ln(2(1-k)) (k > 1/2), straight from the two CDF branches."""
    for r0 in (-3.5, 0.0, 0.25, 7.0):
        for k in (0.01, 0.3, 0.5, 0.7, 0.999):
            for a in (-0.01, -1.0, -5.0):
                t = -a
                want = r0 - t * math.log(2 * k) if k <= 0.5 else r0 + t * math.log(2 * (1 - k))
                x = np.array([r0], dtype=np.float32)
                for f in (O.solve_bisect, O.solve_sorted_scan):
                    got = f(x, k, a)
                    assert abs(got - want) <= 1e-12 * (1 + abs(want)), (f.__name__, r0, k, a, got, want)


def check_all_equal_closed_form():
    """n equal scores c: n sigma((c - b)/t) = k, the n = 1 case at k/n."""
    for n in (2, 7, 64):
        for kk in (0.2, 0.5, 0.9):
            k = kk * n
            a = -0.4
            t = 0.4
            c = 1.375
            want = c - t * math.log(2 * kk) if kk <= 0.5 else c + t * math.log(2 * (1 - kk))
            x = np.full(n, c, dtype=np.float32)
            for f in (O.solve_bisect, O.solve_sorted_scan):
                got = f(x, k, a)
                assert abs(got - want) <= 1e-12 * (1 + abs(want)), (f.__name__, n, k, got, want)


def check_symmetric_half_budget():
    """Scores {x_i} U {-x_i} with k = n/2 give b = 0 exactly, because
    sigma(u) + sigma(-u) = 1."""
    rg = np.random.default_rng(7)
    for n2 in (1, 5, 40):
        h = rg.standard_normal(n2).astype(np.float32)
        x = np.concatenate([h, -h])
        rg.shuffle(x)
        for a in (-0.05, -1.0):
            for f in (O.solve_bisect, O.solve_sorted_scan):
                got = f(x, float(n2), a)
                assert abs(got) <= 1e-12, (f.__name__, n2, a, got)


def check_zero_temperature():
    """Theorem 1: distinct scores, integer k, t -> 0: b -> (r_(k) + r_(k+1))/2.
    Scores on a grid of spacing d: at b = mid the two boundary scores add
    exactly 1 (sigma(u) + sigma(-u) = 1) and every other score is at least
    1.5 d from mid, so |LapSum(mid) - k| <= n/2 e^{-1.5d/t} while the slope
    near mid is at least e^{-0.75d/t}/t: |b - mid| <= n t/2 e^{-0.75d/t}.
    Float64 rounding of the sum (~n 1e-16) adds n 1e-16 / |LapSum'(mid)|
    with |LapSum'(mid)| = e^{-d/(2t)}/t."""
    rg = np.random.default_rng(11)
    d = 0.5
    for _ in range(6):
        n = int(rg.integers(3, 60))
        x = (rg.permutation(n).astype(np.float64) * d + rg.uniform(0, 0.1)).astype(np.float32)
        k = int(rg.integers(1, n))
        mid = O.zero_temperature_threshold(x, k)
        for t in (0.05, 0.03, 0.02, 0.015):
            tol = n * t / 2 * math.exp(-0.75 * d / t) + 1e-14 * n * t * math.exp(d / (2 * t)) + 1e-12
            for f in (O.solve_bisect, O.solve_sorted_scan):
                b = f(x, float(k), -t)
                assert abs(b - mid) <= tol, (f.__name__, n, k, t, b, mid, tol)
        p = O.probs(x, O.solve_sorted_scan(x, float(k), -0.02), -0.02)
        hard = (x.astype(np.float64) > mid).astype(float)
        assert np.max(np.abs(p - hard)) <= 1e-4


def check_equivariance():
    """Shift (r + c => b + c), scale (lambda r, lambda alpha => lambda b) and
    permutation invariance of b, all implied by the definition."""
    rg = np.random.default_rng(3)
    for _ in range(8):
        n = int(rg.integers(2, 120))
        # multiples of 2^-10 below 8 in magnitude: adding 2 and scaling by 4
        # are exact in float32
        x = np.round(np.clip(rg.standard_normal(n), -5, 5) * 1024.0) / 1024.0
        k = float(rg.uniform(0.1, n - 0.1))
        a = -float(rg.uniform(0.05, 2.0))
        for f in (O.solve_bisect, O.solve_sorted_scan):
            b = f(x.astype(np.float32), k, a)
            xs = (x.astype(np.float32) + np.float32(2.0))
            assert abs(f(xs, k, a) - (b + 2.0)) <= 1e-9
            xl = (x.astype(np.float32) * np.float32(4.0))
            assert abs(f(xl, k, 4.0 * a) - 4.0 * b) <= 1e-9 * 4
            perm = rg.permutation(n)
            assert abs(f(x.astype(np.float32)[perm], k, a) - b) <= 1e-10


def check_invariants():
    """sum p = k; 0 <= p <= 1; p strictly increasing in r; tied scores tie."""
    for x, k, a in _rows(12):
        b = O.solve_sorted_scan(x, k, a)
        p = O.probs(x, b, a)
        assert abs(p.sum() - k) <= 1e-9 * max(1.0, k)
        assert np.all(p >= 0) and np.all(p <= 1)
        xd = x.astype(np.float64)
        order = np.argsort(xd, kind="stable")
        ps, xs = p[order], xd[order]
        strict = xs[1:] > xs[:-1]
        assert np.all(ps[1:][strict] >= ps[:-1][strict])
        assert np.all(ps[1:][~strict] == ps[:-1][~strict])


def _decimal_b(x, k, t, digits=40):
    """High-precision bisection of the plain sum with Python's decimal module."""
    getcontext().prec = digits
    xs = [Decimal(float(v)) for v in x]
    K = Decimal(k)
    T = Decimal(t)
    half = Decimal(1) / 2

    def lap(b):
        s = Decimal(0)
        for v in xs:
            u = (v - b) / T
            s += half * u.exp() if u <= 0 else 1 - half * (-u).exp()
        return s

    lo = Decimal(min(float(v) for v in x)) - 50 * T
    hi = Decimal(max(float(v) for v in x)) + 50 * T
    for _ in range(150):
        mid = (lo + hi) / 2
        if lap(mid) > K:
            lo = mid
        else:
            hi = mid
    return float((lo + hi) / 2)


def check_decimal_bruteforce():
    """Tiny cases against a 40-digit bisection written with `decimal`."""
    rg = np.random.default_rng(99)
    for _ in range(10):
        n = int(rg.integers(1, 7))
        x = rg.standard_normal(n).astype(np.float32)
        if n > 2:
            x[1] = x[0]
        k = float(rg.uniform(0.05, n - 0.05))
        t = float(rg.choice([0.01, 0.5, 3.0]))
        want = _decimal_b(x, k, t)
        for f in (O.solve_bisect, O.solve_sorted_scan, O.solve_brent):
            got = f(x, k, -t)
            assert abs(got - want) <= 1e-12 * (1 + abs(want)) + 1e-13 * t, (f.__name__, got, want)


def check_brent(seed_count=12):
    """The library root finder on the plain sum against the two independent
    roots: the 40-digit `decimal` bisection on tiny rows (in
    check_decimal_bruteforce) and, here, float64 bisection of the same sum on
    the mixed rows (ties, heavy tails, t from 1e-3 to 7), and the closed form
    of one score (b = r - t ln(2k) for k <= 1/2, r + t ln(2(1 - k)) above)."""
    for x, k, a in _rows(seed_count):
        b1 = O.solve_bisect(x, k, a)
        b2 = O.solve_brent(x, k, a)
        assert abs(b1 - b2) <= 1e-9 * -a + 1e-12 * abs(b1), (k, a, b1, b2)
    for r0, k, t in ((0.25, 0.3, 0.01), (-3.5, 0.7, 5.0), (7.0, 0.999, 1.0)):
        want = r0 - t * math.log(2 * k) if k <= 0.5 else r0 + t * math.log(2 * (1 - k))
        got = O.solve_brent(np.array([r0], np.float32), k, -t)
        assert abs(got - want) <= 1e-12 * (1 + abs(want)), (r0, k, t, got, want)


def check_certify_root():
    """The sign-change certificate at roots known in closed form: true at the
    root with a margin delta, false when the claimed root is 3 delta off on
    either side (LapSum is strictly decreasing, so then both evaluations sit
    on one side of k).  Roots: one score (b = r - t ln(2k)), the symmetric
    row {x, -x} at k = n/2 (b = 0), and n equal scores c (b = c - t ln(2k/n)
    for k <= n/2)."""
    rg = np.random.default_rng(4)
    x = rg.standard_normal(500).astype(np.float32)
    cases = [
        (np.array([0.5], np.float32), 0.2, -0.3, 0.5 - 0.3 * math.log(0.4)),
        (np.concatenate([x, -x]), 500.0, -0.05, 0.0),
        (np.full(64, 1.25, np.float32), 8.0, -2.0, 1.25 - 2.0 * math.log(2 * 8.0 / 64)),
    ]
    for r, k, a, b in cases:
        t = -a
        for delta in (1e-6 * t, 1e-3 * t):
            assert O.certify_root(r, k, a, b, delta), (k, a, b, delta)
            assert not O.certify_root(r, k, a, b + 3 * delta, delta), (k, a, b, delta, "+")
            assert not O.certify_root(r, k, a, b - 3 * delta, delta), (k, a, b, delta, "-")


def check_vjp_fd(configs=((2, 32, 4, -1.0), (1, 64, 8, -0.5), (2, 64, 16, -2.0)), tol=1e-8):
    """Eq. (5) against centred finite differences (the gradcheck protocol)."""
    worst = 0.0
    for ci, (B, n, k, a) in enumerate(configs):
        rg = np.random.default_rng([77, ci])
        for _row in range(B):
            x = rg.standard_normal(n)
            g = rg.standard_normal(n)
            b = O.solve_bisect(x, k, a)
            an = O.vjp(x, b, a, g)
            fd = O.fd_vjp(x, k, a, g)
            rel = np.max(np.abs(an - fd)) / np.max(np.abs(fd))
            worst = max(worst, rel)
    assert worst <= tol, worst
    return worst


def check_vjp_invariants():
    """Derived from Eq. (5): sum of the VJP is zero (b absorbs a uniform shift),
    a constant cotangent gives zero, and the Jacobian is symmetric."""
    rg = np.random.default_rng(5)
    for _ in range(6):
        n = int(rg.integers(2, 80))
        x = rg.standard_normal(n)
        k = float(rg.uniform(0.5, n - 0.5))
        a = -float(rg.uniform(0.1, 2.0))
        b = O.solve_bisect(x, k, a)
        g = rg.standard_normal(n)
        v = O.vjp(x, b, a, g)
        assert abs(v.sum()) <= 1e-12 * (1 + np.abs(v).sum())
        assert np.max(np.abs(O.vjp(x, b, a, np.full(n, 3.25)))) <= 1e-14
        u = rg.standard_normal(n)
        assert abs(np.dot(u, O.vjp(x, b, a, g)) - np.dot(g, O.vjp(x, b, a, u))) <= 1e-12


def check_params_fd(cases=((24, 6.0, -1.0), (40, 13.5, -0.3), (64, 3.25, -2.0)), tol=1e-6):
    """dL/dk and dL/dalpha against centred finite differences of <g, p> in k
    and alpha, each threshold re-solved by its definition."""
    worst = 0.0
    for ci, (n, k, a) in enumerate(cases):
        rg = np.random.default_rng([91, ci])
        x = rg.standard_normal(n)
        g = rg.standard_normal(n)
        b = O.solve_bisect(x, k, a)
        got = O.vjp_params(x, b, a, g)
        fd = O.fd_params(x, k, a, g)
        for an, nu in zip(got, fd):
            rel = abs(an - nu) / max(abs(nu), 1e-3)
            worst = max(worst, rel)
    assert worst <= tol, worst
    return worst


def check_params_closed_forms():
    """Cases with closed forms: one score (p = k whatever alpha), all scores
    equal (p = k/n), and a constant cotangent c (<c, p> = c k): the gradients
    are (mean g, 0), (mean g, 0) and (c, 0)."""
    rg = np.random.default_rng(17)
    gk, ga = O.vjp_params(np.array([0.7]), O.solve_bisect(np.array([0.7]), 0.3, -0.5), -0.5,
                          np.array([2.5]))
    assert abs(gk - 2.5) <= 1e-15 and abs(ga) <= 1e-15
    for n in (2, 9, 50):
        x = np.full(n, -1.25)
        g = rg.standard_normal(n)
        k = 0.37 * n
        gk, ga = O.vjp_params(x, O.solve_bisect(x, k, -0.8), -0.8, g)
        assert abs(gk - g.mean()) <= 1e-14 * (1 + np.abs(g).max()) and abs(ga) <= 1e-14
    for _ in range(5):
        n = int(rg.integers(3, 60))
        x = rg.standard_normal(n)
        a = -float(rg.uniform(0.05, 3.0))
        k = float(rg.uniform(0.5, n - 0.5))
        gk, ga = O.vjp_params(x, O.solve_bisect(x, k, a), a, np.full(n, -1.5))
        assert abs(gk + 1.5) <= 1e-14 and abs(ga) <= 1e-12


def check_params_scale_identity():
    """p(c r, k, c alpha) = p(r, k, alpha) for c > 0 (Eq. (1) depends on
    (r - b)/alpha only), so d/dc at c = 1 gives
    alpha dL/dalpha = -<r, grad_r L>, tying dL/dalpha to Eq. (5)."""
    rg = np.random.default_rng(23)
    for _ in range(6):
        n = int(rg.integers(2, 90))
        x = rg.standard_normal(n) * rg.uniform(0.5, 4.0) + rg.uniform(-3, 3)
        a = -float(rg.uniform(0.05, 3.0))
        k = float(rg.uniform(0.5, n - 0.5))
        g = rg.standard_normal(n)
        b = O.solve_bisect(x, k, a)
        _, ga = O.vjp_params(x, b, a, g)
        rhs = -float(np.dot(x, O.vjp(x, b, a, g)))
        scale = float(np.dot(np.abs(x), np.abs(O.vjp(x, b, a, np.abs(g))))) + 1e-300
        assert abs(a * ga - rhs) <= 1e-12 * max(scale, abs(rhs), 1.0), (a * ga, rhs)


def check_dftopk_fd(cases=((64, 8, -0.5), (48, 24, -0.05), (33, 1, -2.0), (33, 32, -1.0))):
    """The DFTopK vector-Jacobian product against centred finite differences
    of <g, p(r)>.  The operator reads float32 scores, so the scores are
    float32 values in (-2, 2) and the step is 2^-14, exact in float32 there;
    the scores are drawn until no two lie within 8 steps, so no pair swaps
    and the boundary pair stays the same."""
    eps = 2.0 ** -14
    for ci, (n, k, a) in enumerate(cases):
        rg = np.random.default_rng([31, ci])
        while True:
            x = rg.uniform(-2.0, 2.0, n).astype(np.float32).astype(np.float64)
            if np.min(np.diff(np.sort(x))) > 8 * eps:
                break
        g = rg.standard_normal(n)
        an = O.dftopk_vjp(x, k, a, g)
        fd = np.empty(n)
        for i in range(n):
            xp = x.copy(); xp[i] += eps
            xm = x.copy(); xm[i] -= eps
            fd[i] = (np.dot(g, O.dftopk(xp, k, a)[0]) - np.dot(g, O.dftopk(xm, k, a)[0])) / (2 * eps)
        rel = np.max(np.abs(an - fd)) / np.max(np.abs(fd))
        # centred differences err by h^2/6 times the third derivative,
        # at most 1/(8 t^2) of the first for the logistic step
        assert rel <= 1e-6, (ci, rel)


def check_dftopk_midpoint_is_the_zero_temperature_threshold():
    """Theorem 1: LapSum's threshold tends to the midpoint of r_(k), r_(k+1)
    as t -> 0; DFTopK fixes its threshold there at every t."""
    rg = np.random.default_rng(41)
    for _ in range(8):
        n = int(rg.integers(2, 300))
        k = int(rg.integers(1, n))
        x = rg.standard_normal(n).astype(np.float32)
        assert O.dftopk(x, k, -0.3)[1] == O.zero_temperature_threshold(x, k)


def check_dftopk_budget_table(rows):
    """Table budget, DFTopK row: the relative mass error |sum p - k|/k on
    Gaussian scores with k = n/16, alpha = -1, within the sampling spread of
    one draw (4 standard deviations of the mean of the logistic step, plus
    the table's rounding)."""
    for n, want in rows:
        x = np.random.default_rng([51, n]).standard_normal(n).astype(np.float32)
        p = O.dftopk(x, n // 16, -1.0)[0]
        got = abs(math.fsum(p) - n // 16) / (n // 16)
        spread = 16.0 * 0.3 / math.sqrt(n) * 4.0 + 0.005
        assert abs(got - want) <= spread, (n, got, want, spread)


def check_desc_order():
    """Descending by value; equal values keep ascending index; -0.0 after +0.0."""
    rg = np.random.default_rng(1)
    x = rg.integers(-5, 5, 500).astype(np.float32) * np.float32(0.5)
    x[10] = np.float32(-0.0)
    x[20] = np.float32(0.0)
    perm = O.desc_order(x)
    want = sorted(range(x.size), key=lambda i: (-float(x[i]), i))
    # the two orders differ only in where the signed zeros fall
    zeros = {i for i in range(x.size) if x[i] == 0}
    assert [i for i in perm if i not in zeros] == [i for i in want if i not in zeros]
    zpos = [int(np.nonzero(perm == i)[0][0]) for i in (10, 20)]
    assert zpos[1] < zpos[0]  # +0.0 (index 20) before -0.0 (index 10)
    assert np.all(np.diff(x[perm].astype(np.float64)) <= 0)


def check_bracket_ranks():
    """Eq. (8) pinned by what it must achieve: the normal-approximation
    coverage Pr(j <= C <= l-1) >= 1 - 2 Phi(-z) (minus the Berry-Esseen slack)
    for C ~ Bin(K, q), with a width no more than 2 z sd + 2."""
    from scipy.stats import binom, norm
    for (n, k, K, z) in [(10**7, 2000.0, 46416, 5.16), (10**8, 20000.0, 10**5, 5.16),
                         (20000, 5000.0, 700, 2.0), (1000, 62.5, 100, 1.0),
                         (10**6, 1000.0, 10**4, 3.0)]:
        j, l, q = O.bracket_ranks(n, k, K, z)
        assert abs(q - (n - k) / n) < 1e-15
        sd = math.sqrt(K * q * (1 - q))
        cover = binom.cdf(min(l, K + 1) - 1, K, q) - binom.cdf(j - 1, K, q)
        assert cover >= 1 - 2 * norm.cdf(-z) - 3.0 / math.sqrt(K * q * (1 - q)), (n, cover)
        assert (l - j) <= 2 * z * sd + 2
        assert j <= K * q <= l


def check_partition_definition():
    """Suppl. B set definitions at exact float32 boundary values and Eq. (7)."""
    x = np.array([1.0, 2.0, 3.0, 2.0, 5.0, 0.5, 3.0], dtype=np.float32)
    part = O.partition(x, 2.0, 3.0, 0.5)
    assert (part.n_L, part.n_M, part.n_R) == (2, 2, 3)
    assert list(part.m_idx) == [1, 3]
    want_L = math.exp(-(2.0 - 1.0) / 0.5) + math.exp(-(2.0 - 0.5) / 0.5)
    want_R = 2 * math.exp(0.0) + math.exp(-(5.0 - 3.0) / 0.5)
    assert abs(part.T_L - want_L) < 1e-15 and abs(part.T_R - want_R) < 1e-15


def check_bracket_equals_full():
    """Suppl. B exactness: the bracketed solve reproduces the definition."""
    cases = [("normal", 20000, 5000.0, -0.3, 700, 2.0),
             ("laplace_abs", 30000, 2.0, -0.01, 965, 5.16),
             ("levels16", 20000, 1250.0, -1.0, 737, 5.16),
             ("clusters3", 25000, 12000.0, -0.05, 855, 3.0),
             ("cauchy", 20000, 1250.0, -1.0, 737, 5.16),
             ("student2", 20000, 19000.0, -0.2, 700, 1.0)]
    for ci, (dist, n, k, a, K, z) in enumerate(cases):
        x = W.random_case(ci, n, dist=dist, ties=0.01)[0]
        eps = W.laplace_noise([55, ci], K, -a)
        p, b, info, ms = O.bracketed_forward(x, k, a, eps, z=z)
        bb = O.solve_bisect(x, k, a)
        assert abs(b - bb) <= 1e-9 * -a + 1e-12 * abs(bb), (dist, b, bb, info)
        if not info.fell_back:
            part = O.partition(x, info.a_L, info.a_R, -a)
            assert set(ms.tolist()) == set(part.m_idx.tolist())
            assert info.lap_aR <= k <= info.lap_aL


def check_forced_widening():
    """Noise tables shifted far from zero make the first bracket miss b; the
    validated path must widen the failing side and still return the exact b
    (Suppl. C, Expected Linear Runtime; Algorithm 1 step 4)."""
    n, k, a, K = 20000, 1250.0, -0.5, 737
    x = W.random_case(4, n, dist="normal")[0]
    bb = O.solve_bisect(x, k, a)
    base = W.laplace_noise([56], K, 0.5)
    for shift, attempts, fell in ((0.0, 1, 0), (3.0, 3, 0), (-3.0, 3, 0), (30.0, 3, 1)):
        p, b, info, ms = O.bracketed_forward(x, k, a, base + np.float32(shift), z=5.16)
        assert abs(b - bb) <= 1e-9, (shift, b, bb, info)
        assert (info.attempts, info.fell_back) == (attempts, fell), (shift, info)
        if not fell:
            assert info.a_L <= b <= info.a_R
    # a zero-width bracket never certifies: three attempts, then the full sort
    xc = np.full(n, 1.0, dtype=np.float32)
    xc[::3] = 2.0
    p, b, info, ms = O.bracketed_forward(xc, 100.5, -0.01, np.zeros(K, np.float32), z=1e-9)
    assert info.a_L == info.a_R and info.fell_back == 1 and info.attempts == 3
    assert abs(b - O.solve_bisect(xc, 100.5, -0.01)) <= 1e-10
    # no room for M: straight to the full sort
    p, b, info, ms = O.bracketed_forward(x, k, a, base, z=5.16, m_capacity=10)
    assert info.m_overflow == 1 and info.fell_back == 1 and info.attempts == 1
    assert abs(b - bb) <= 1e-9


def check_sampler_and_order_statistic():
    """The systematic sampler reads r[s * floor(n/K)] and adds the noise in
    float32; y_(j) is the j-th smallest, 1-based, infinite outside 1..K."""
    r = np.arange(1000, dtype=np.float32)
    y = O.systematic_sample(r, np.zeros(7, np.float32))
    assert y.tolist() == [0.0, 142.0, 284.0, 426.0, 568.0, 710.0, 852.0]
    y = O.systematic_sample(np.full(10, 1.0, np.float32), np.full(5, 2.0 ** -30, np.float32))
    assert np.all(y == np.float32(1.0))          # 1 + 2^-30 rounds to 1 in float32
    v = np.array([5.0, -1.0, 3.0, 3.0, 0.5], np.float32)
    assert [O.order_statistic(v, j) for j in (1, 2, 3, 4, 5)] == [-1.0, 0.5, 3.0, 3.0, 5.0]
    assert O.order_statistic(v, 0) == -math.inf and O.order_statistic(v, 6) == math.inf
    # the i.i.d. sampler at the strided indices is the systematic one, and it
    # reads the indices it is given, in their order
    rg = np.random.default_rng(8)
    x = rg.standard_normal(1000).astype(np.float32)
    e = rg.laplace(0.0, 0.1, 7).astype(np.float32)
    assert np.array_equal(O.iid_sample(x, np.arange(7) * 142, e), O.systematic_sample(x, e))
    assert O.iid_sample(r, [999, 3, 3], np.zeros(3, np.float32)).tolist() == [999.0, 3.0, 3.0]


def check_widen_rule():
    """One-sided doubling with simultaneous assignment."""
    assert O.widen(1.0, 2.0, "right") == (2.0, 4.0)
    assert O.widen(1.0, 2.0, "left") == (-1.0, 1.0)
    assert O.widen(-math.inf, 2.0, "right") == (2.0, math.inf)
    assert O.widen(1.0, math.inf, "left") == (-math.inf, 1.0)


def check_coverage_theorem(trials=1500):
    """Theorem 2 with i.i.d. draws: Pr(y_(j) <= b < y_(l)) = Pr(j <= C <= l-1),
    C ~ Bin(K, q).  Small z so that misses are frequent enough to count."""
    from scipy.stats import binom
    rg = np.random.default_rng(2024)
    n, k, a = 2000, 300.0, -0.2
    t = -a
    x = rg.standard_normal(n).astype(np.float32)
    b = O.solve_bisect(x, k, a)
    for K, z in ((200, 0.5), (400, 1.0)):
        j, l, q = O.bracket_ranks(n, k, K, z)
        want = binom.cdf(l - 1, K, q) - binom.cdf(j - 1, K, q)
        hits = 0
        for _ in range(trials):
            y = O.iid_sample(x, rg.integers(0, n, K), rg.laplace(0.0, t, K).astype(np.float32))
            aL, aR = O.order_statistic(y, j), O.order_statistic(y, l)
            hits += (aL <= b < aR)
        freq = hits / trials
        sd = math.sqrt(want * (1 - want) / trials)
        assert abs(freq - want) <= 4.5 * sd + 1e-3, (K, z, freq, want)


def check_budget_table(sizes=(1000, 10000, 100000)):
    """Table budget: float32 p from the exact threshold keeps |sum p - k|/k
    below 1e-5 (k = n/16, alpha = -1, Gaussian scores)."""
    rg = np.random.default_rng(8)
    for n in sizes:
        x = rg.standard_normal(n).astype(np.float32)
        k = n / 16.0
        b = O.solve_sorted_scan(x, k, -1.0)
        p32 = O.probs(x, b, -1.0).astype(np.float32)
        assert O.budget_error(p32, k) / k < 1e-5


def check_splitmix64(rows):
    """The generator against its published outputs (tests/golden)."""
    for seed, want in rows:
        assert O.splitmix64(seed, len(want)) == list(want), seed


def check_counter_noise():
    """The default kernel noise is Laplace(0, t): a Kolmogorov-Smirnov test
    against scipy's Laplace distribution (a wrong scale, sign or branch
    fails it at these sizes), its sign follows the top bit of the generator
    output (u >= 1/2 exactly when bit 63 is set), and the draws are the
    generator's in order (a different seed or a shifted counter gives
    different draws)."""
    from scipy import stats
    for seed, t in ((0, 0.01), (7, 1.0), ((1 << 64) - 1, 0.05)):
        x = O.counter_laplace_noise(seed, 20000, t)
        assert x.dtype == np.float32 and x.shape == (20000,)
        ks = stats.kstest(x.astype(np.float64), stats.laplace(loc=0.0, scale=t).cdf)
        assert ks.pvalue > 1e-3, (seed, t, ks)
        top = np.array([v >> 63 for v in O.splitmix64(seed, 20000)])
        assert np.array_equal(top == 1, x >= 0), seed
    a = O.counter_laplace_noise(3, 100, 0.5)
    assert np.array_equal(O.counter_laplace_noise(3, 50, 0.5), a[:50])
    assert not np.array_equal(O.counter_laplace_noise(4, 100, 0.5), a)
