"""Float64 CPU oracle for the exact-budget LapSum soft top-k ("Fast LapSum").

TEST INFRASTRUCTURE ONLY.  The test-suite, the smoke check of the build entry
point and the benchmark's CPU-baseline leg are the only code allowed to import,
call or execute anything in this package.  The HIP library never calls it, and
the two share no code: no kernels, helpers, tables or pre/post-processing.

Plain, slow and written to be checked against the paper by eye.  Arithmetic is
IEEE float64 unless a step of the method is defined in float32 (the noised
sample of the bracket, Suppl. C); scores are promoted from float32 exactly.

Notation (the paper's): scores r in R^n, budget k in (0, n), temperature
alpha < 0 and t = |alpha| = -alpha, Laplace CDF sigma, threshold b with
LapSum(b) = sum_i sigma((b - r_i)/alpha) = k (Eq. (1), Suppl. A).

What each function restates
---------------------------
laplace_cdf            Eq. (3) / Suppl. A, the Laplace CDF.
lapsum                 Suppl. A, the budget function LapSum(b).
solve_bisect           the definition: the unique root of LapSum(b) = k,
                       by bisection on the plain sum (the per-query solver
                       that §5 uses as its baseline).
solve_brent            the same root by a library root finder on the plain
                       sum (for n where 200 bisection sums are too slow).
certify_root           sign change of LapSum(b) - k around b.
solve_sorted_scan      Suppl. A / §1 / §3: sort descending, prefix/suffix
                       exponential scans give the node curve LapSum(r_(i)),
                       index lookup, closed-form root of the two-exponential
                       equation inside the interval.
probs                  Eq. (1): p_i = sigma((b - r_i)/alpha).
vjp                    Eq. (5): (grad_r p)^T g = f * (g - <g, q>).
fd_vjp                 centred finite differences (Suppl. F, Table gradcheck
                       protocol).
vjp_params             §5 (the attack trains k and alpha): dL/dk and dL/dalpha
                       by implicit differentiation of Eq. (1) (a reading; the
                       paper gives no formula).
fd_params              centred finite differences of <g, p> in k and alpha.
bracket_ranks          Eq. (8): j = floor(Kq - z sqrt(Kq(1-q))),
                       l = ceil(Kq + z sqrt(Kq(1-q))), q = (n-k)/n.
splitmix64             the counter-based generator behind the default
                       kernel noise (its published definition).
counter_laplace_noise  the default kernel noise: Laplace(0, t) by the
                       inverse CDF of SplitMix64 uniforms.
systematic_sample      §4 / Suppl. C remark (iii): strided view plus cached
                       kernel noise, y_s = r_{s*stride} + eps_s.
iid_sample             Suppl. C, Theorem 2: uniform draws with replacement
                       (indices given) plus kernel noise.
partition              Suppl. B: L, M, R sets and the tail sums of Eq. (7).
solve_in_bracket       Suppl. B: LapSum(b) = |R| + 1/2 S_L e^{(b-a_L)/alpha}
                       - 1/2 S_R e^{(a_R-b)/alpha} + sum_M sigma(.), solved on
                       the sorted middle set with the tails as carries.
widen                  Suppl. C "Expected Linear Runtime": one-sided doubling.
bracketed_forward      Algorithm 1 (Sample-bracketed soft top-k) with the
                       validated path: certify, widen, fall back.
zero_temperature_threshold  Theorem 1: the midpoint of r_(k), r_(k+1).
dftopk, dftopk_vjp     the DFTopK comparator (§2, Suppl. "Comparison with
                       DFTopK"): logistic step at that fixed midpoint, and
                       its vector-Jacobian product.

Readings of the paper (where it is silent or ambiguous) are listed in the
repository's design notes; the ones that change a number are repeated at the
function that takes them.

Parity status: every function above is pinned by CPU tests against closed
forms, invariants, brute force or the definition, except the coverage rate
of the systematic sampler (Table robustness), which has no closed form and is
"parity unpinned".
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

F64 = np.float64

__all__ = [
    "laplace_cdf", "lapsum", "initial_bracket", "solve_bisect", "solve_brent",
    "certify_root", "desc_keys", "desc_order", "solve_sorted_scan", "probs",
    "vjp", "vjp_params", "forward", "fd_vjp", "fd_params", "bracket_ranks", "systematic_sample",
    "iid_sample", "dftopk", "dftopk_vjp", "splitmix64", "counter_laplace_noise",
    "order_statistic", "partition", "solve_in_bracket", "widen",
    "BracketInfo", "bracketed_forward", "zero_temperature_threshold",
    "budget_error",
]

_CHUNK = 1 << 22


# --------------------------------------------------------------------------
# The operator
# --------------------------------------------------------------------------

def laplace_cdf(u):
    """sigma(u) = 1/2 e^u for u <= 0 and 1 - 1/2 e^{-u} for u > 0 (Eq. (3))."""
    u = np.asarray(u, dtype=F64)
    out = np.empty_like(u)
    neg = u <= 0.0
    out[neg] = 0.5 * np.exp(u[neg])
    pos = ~neg
    out[pos] = 1.0 - 0.5 * np.exp(-u[pos])
    return out


def _as_f64(r) -> np.ndarray:
    return np.asarray(r).astype(F64, copy=False).ravel()


def lapsum(r, b: float, t: float) -> float:
    """LapSum(b) = sum_i sigma((b - r_i)/alpha) = sum_i sigma((r_i - b)/t).

    Suppl. A.  With alpha < 0 the two forms are the same number.  The sum is
    NumPy's pairwise sum inside chunks of 4M terms and an exactly rounded
    `math.fsum` over the chunk sums.
    """
    r = _as_f64(r)
    parts = []
    for a in range(0, r.size, _CHUNK):
        parts.append(float(np.sum(laplace_cdf((r[a:a + _CHUNK] - b) / t))))
    return math.fsum(parts)


def initial_bracket(r, k: float, t: float) -> tuple[float, float]:
    """lo, hi with LapSum(lo) > k > LapSum(hi) for 0 < k < n.

    At b = lo every score is at least r_min - lo above b, so
    LapSum(lo) >= n - n/2 e^{-(r_min-lo)/t} > k once
    r_min - lo >= t (ln(n / (2(n-k))) + 1); symmetrically for hi.
    """
    r = _as_f64(r)
    n = r.size
    lo = float(r.min()) - t * (max(0.0, math.log(n / (2.0 * (n - k)))) + 1.0)
    hi = float(r.max()) + t * (max(0.0, math.log(n / (2.0 * k))) + 1.0)
    return lo, hi


def _check(r, k, alpha):
    r = _as_f64(r)
    if r.size < 1:
        raise ValueError("need n >= 1")
    if not np.all(np.isfinite(r)):
        raise ValueError("scores must be finite")
    if not (math.isfinite(alpha) and alpha < 0.0):
        raise ValueError("alpha must be finite and < 0")
    if not (math.isfinite(k) and 0.0 < k < r.size):
        raise ValueError("k must lie in (0, n)")
    return r, -float(alpha)


def solve_bisect(r, k: float, alpha: float, iters: int = 200) -> float:
    """The threshold by its definition: the root of LapSum(b) = k.

    LapSum is strictly decreasing in b (each sigma((r_i - b)/t) is), so the
    root is unique.  Bisection on the plain sum, as the prior per-query
    solvers do (§1, §5), for up to `iters` halvings or until the interval
    cannot shrink in float64.
    """
    r, t = _check(r, k, alpha)
    lo, hi = initial_bracket(r, k, t)
    for _ in range(iters):
        mid = 0.5 * (lo + hi)
        if mid <= lo or mid >= hi:
            break
        if lapsum(r, mid, t) > k:
            lo = mid
        else:
            hi = mid
    return 0.5 * (lo + hi)


def solve_brent(r, k: float, alpha: float) -> float:
    """The same root as `solve_bisect`, by Brent's method on the plain sum."""
    from scipy.optimize import brentq

    r, t = _check(r, k, alpha)
    lo, hi = initial_bracket(r, k, t)
    return float(brentq(lambda b: lapsum(r, b, t) - k, lo, hi,
                        xtol=1e-14 * t, rtol=4.0 * np.finfo(F64).eps, maxiter=500))


def certify_root(r, k: float, alpha: float, b: float, delta: float) -> bool:
    """True iff LapSum(b - delta) > k > LapSum(b + delta), i.e. the true root
    lies within delta of b (LapSum is strictly decreasing)."""
    r, t = _check(r, k, alpha)
    return lapsum(r, b - delta, t) > k > lapsum(r, b + delta, t)


# --------------------------------------------------------------------------
# Sorting order (reading: descending by value, ties by ascending index)
# --------------------------------------------------------------------------

def desc_keys(r32) -> np.ndarray:
    """uint32 keys whose ascending order is the descending order of the
    float32 scores.  Ascending map: non-negative floats get the sign bit set,
    negative floats are bit-inverted; the descending key is its complement.
    -0.0 therefore sorts after +0.0 (equal values, distinct keys)."""
    bits = np.ascontiguousarray(r32, dtype=np.float32).view(np.uint32)
    neg = (bits >> np.uint32(31)) != 0
    asc = np.where(neg, ~bits, bits | np.uint32(0x80000000))
    return ~asc


def desc_order(r32) -> np.ndarray:
    """Stable permutation: position i holds the original index of the i-th
    largest score; equal keys keep ascending original index."""
    return np.argsort(desc_keys(r32), kind="stable")


# --------------------------------------------------------------------------
# Closed form on a sorted array (Suppl. A, Suppl. B)
# --------------------------------------------------------------------------

def _node_curve(s: np.ndarray, t: float, n_above: int, above, below):
    """Node values of the budget curve on a descending array s.

    above = None or (anchor u, sum A): scores ranked before s (all >= u >= s_1)
            summarised as A = sum exp(-(r - u)/t);
    below = None or (anchor v, sum B): scores ranked after s (all <= v <= s_m)
            summarised as B = sum exp(-(v - r)/t).
    Returns (logP, logQ, N) with, for position i (1-based, global rank
    n_above + i):
        P_i = sum_{rank <= i} exp(-(r - s_i)/t)           (prefix, >= 1)
        Q_i = sum_{rank >= i} exp(-(s_i - r)/t)           (suffix, >= 1)
        E_i = Q_{i+1} exp(-(s_i - s_{i+1})/t) or B exp(-(s_i - v)/t) at the end
        N_i = LapSum(s_i) = n_above + i - P_i/2 + E_i/2
    The three-group split at b = s_i (ranks before, equal, after) of Suppl. A.
    Cumulative sums are taken in the log domain (np.logaddexp.accumulate), so
    each term is formed relative to its own node and nothing overflows.
    """
    m = s.size
    x = -s / t
    if above is not None and above[1] > 0.0:
        x0 = math.log(above[1]) - above[0] / t
        cum = np.logaddexp.accumulate(np.concatenate(([x0], x)))[1:]
    else:
        cum = np.logaddexp.accumulate(x)
    logP = cum + s / t
    y = s / t
    if below is not None and below[1] > 0.0:
        y0 = math.log(below[1]) + below[0] / t
        rcum = np.logaddexp.accumulate(np.concatenate(([y0], y[::-1])))[1:][::-1]
    else:
        rcum = np.logaddexp.accumulate(y[::-1])[::-1]
    logQ = rcum - s / t
    E = np.empty(m, dtype=F64)
    if m > 1:
        E[:-1] = np.exp(logQ[1:] - (s[:-1] - s[1:]) / t)
    if below is not None and below[1] > 0.0:
        E[-1] = below[1] * math.exp(-(s[-1] - below[0]) / t)
    else:
        E[-1] = 0.0
    i = np.arange(1, m + 1, dtype=F64)
    N = n_above + i - 0.5 * np.exp(logP) + 0.5 * E
    return logP, logQ, N


def _gap_root(k: float, t: float, c_up: float, up, down) -> float:
    """Root of LapSum(b) = k on one interval of the curve.

    For b between the upper knot u and the lower knot v (v <= b <= u) the
    scores split into the c_up scores ranked above (summary (u, A), A =
    sum exp(-(r-u)/t)) and those below (summary (v, B), B = sum exp(-(v-r)/t)):
        LapSum(b) = c_up - A/2 e^{-(u-b)/t} + B/2 e^{-(b-v)/t}
    (the two-exponential form that makes the local root closed form, §3).
    With y = e^{(u-b)/t} and E = B e^{-(u-v)/t} this is
        E y^2 - 2 (k - c_up) y - A = 0,
    solved in the log domain.  up or down is None when its sum is zero (no
    scores, or all of them saturated); the c_up scores above still count.
    """
    if up is None and down is None:
        raise ValueError("empty problem")
    if up is None:
        # LapSum(b) = c_up + B/2 e^{-(b-v)/t}
        v, lnB = down
        return v + t * (lnB - math.log(2.0 * (k - c_up)))
    if down is None:
        u, lnA = up
        return u - t * (lnA - math.log(2.0 * (c_up - k)))
    u, lnA = up
    v, lnB = down
    g = (u - v) / t
    lnE = lnB - g
    c = k - c_up
    if c > 0.0:
        # D = sqrt(c^2 + A E); ln y = ln(c + D) - ln E
        lnAE = lnA + lnE
        lnD = 0.5 * np.logaddexp(2.0 * math.log(c), lnAE)
        lny = float(np.logaddexp(math.log(c), lnD)) - lnE
    elif c < 0.0:
        lnAE = lnA + lnE
        lnD = 0.5 * np.logaddexp(2.0 * math.log(-c), lnAE)
        lny = lnA - float(np.logaddexp(math.log(-c), lnD))
    else:
        lny = 0.5 * (lnA - lnE)
    lny = min(max(lny, 0.0), g)
    return u - t * lny


def solve_sorted_scan(r, k: float, alpha: float) -> float:
    """Threshold by the full-sort closed form (§1, §3, Suppl. A).

    1. sort the scores descending, s_1 >= ... >= s_n;
    2. prefix and suffix exponential scans give the node values
       N_i = LapSum(s_i), non-decreasing in i;
    3. index lookup m = #{i : N_i <= k}, so b lies in [s_{m+1}, s_m];
    4. closed-form root of the two-exponential equation in that interval
       (m = 0: above s_1; m = n: below s_n).
    """
    r, t = _check(r, k, alpha)
    r32 = np.asarray(r, dtype=np.float32)
    s = r[desc_order(r32)]
    return _solve_on_sorted(s, k, t, 0, None, None)


def _solve_on_sorted(s, k, t, n_above, above, below) -> float:
    m_len = s.size
    if m_len == 0:
        up = None if above is None or above[1] <= 0.0 else (above[0], math.log(above[1]))
        dn = None if below is None or below[1] <= 0.0 else (below[0], math.log(below[1]))
        return _gap_root(k, t, float(n_above), up, dn)
    logP, logQ, N = _node_curve(s, t, n_above, above, below)
    m = int(np.count_nonzero(N <= k))
    if m == 0:
        up = None if above is None or above[1] <= 0.0 else (above[0], math.log(above[1]))
        dn = (float(s[0]), float(logQ[0]))
        return _gap_root(k, t, float(n_above), up, dn)
    if m == m_len:
        up = (float(s[-1]), float(logP[-1]))
        dn = None if below is None or below[1] <= 0.0 else (below[0], math.log(below[1]))
        return _gap_root(k, t, float(n_above + m_len), up, dn)
    up = (float(s[m - 1]), float(logP[m - 1]))
    dn = (float(s[m]), float(logQ[m]))
    return _gap_root(k, t, float(n_above + m), up, dn)


# --------------------------------------------------------------------------
# Outputs and backward
# --------------------------------------------------------------------------

def probs(r, b: float, alpha: float) -> np.ndarray:
    """p_i = sigma((b - r_i)/alpha) (Eq. (1)), float64."""
    t = -float(alpha)
    return laplace_cdf((_as_f64(r) - b) / t)


def vjp(r, b: float, alpha: float, g) -> np.ndarray:
    """(grad_r p)^T g = f * (g - <g, q>), q = f / sum f,
    f_i = exp(-|b - r_i|/|alpha|) / (2|alpha|)   (Eq. (5)).
    Reading: when sum f is zero in float64 the product is taken as zero."""
    t = -float(alpha)
    r = _as_f64(r)
    g = _as_f64(g)
    f = np.exp(-np.abs(b - r) / t) / (2.0 * t)
    sf = math.fsum(f)
    if sf == 0.0:
        return np.zeros_like(r)
    gq = math.fsum(g * f) / sf
    return f * (g - gq)


def forward(r, k: float, alpha: float, method: str = "bisect"):
    """(p, b) for one row."""
    if method == "bisect":
        b = solve_bisect(r, k, alpha)
    elif method == "brent":
        b = solve_brent(r, k, alpha)
    elif method == "scan":
        b = solve_sorted_scan(r, k, alpha)
    else:
        raise ValueError(method)
    return probs(r, b, alpha), b


def fd_vjp(r, k: float, alpha: float, g, eps: float = 1e-5) -> np.ndarray:
    """Centred finite differences of <g, p(r)> in float64, one coordinate at a
    time (the protocol of Table gradcheck)."""
    r = _as_f64(r).copy()
    g = _as_f64(g)
    out = np.empty_like(r)
    for i in range(r.size):
        x = r[i]
        r[i] = x + eps
        fp = float(np.dot(g, probs(r, solve_bisect(r, k, alpha), alpha)))
        r[i] = x - eps
        fm = float(np.dot(g, probs(r, solve_bisect(r, k, alpha), alpha)))
        r[i] = x
        out[i] = (fp - fm) / (2.0 * eps)
    return out


def vjp_params(r, b: float, alpha: float, g) -> tuple[float, float]:
    """(dL/dk, dL/dalpha) for L = <g, p> with b tied to (k, alpha) by Eq. (1).

    §5 (exact-budget adversarial examples) trains both the budget k and the
    temperature alpha; the paper states no formula, so this is a reading:
    implicit differentiation of sum_i sigma((r_i - b)/t) = k, t = -alpha.
    With s_i = exp(-|r_i - b|/t)/2 (so that dp_i/db = -s_i/t, the f of
    Eq. (5) times t) and u_i = (r_i - b)/t:
        db/dk = -t / sum s,   dp_i/dk = s_i / sum s,
        db/dt = -t sum s u / sum s,   dp_i/dt = -(s_i/t)(u_i - sum s u / sum s),
    so with F = sum s, G = sum s g, U = sum s u, H = sum s g u
        dL/dk = G / F,   dL/dalpha = -dL/dt = (H - (U/F) G) / t.
    Both are taken as zero when F is zero in float64 (as in `vjp`)."""
    t = -float(alpha)
    r = _as_f64(r)
    g = _as_f64(g)
    u = (r - b) / t
    s = 0.5 * np.exp(-np.abs(u))
    F = math.fsum(s)
    if F == 0.0:
        return 0.0, 0.0
    G = math.fsum(s * g)
    U = math.fsum(s * u)
    H = math.fsum(s * g * u)
    return G / F, (H - (U / F) * G) / t


def fd_params(r, k: float, alpha: float, g, eps: float = 1e-6) -> tuple[float, float]:
    """Centred finite differences of <g, p(k, alpha)> in k and in alpha, each
    re-solving the threshold by its definition."""
    def loss(kk, aa):
        return float(np.dot(_as_f64(g), probs(r, solve_bisect(r, kk, aa), aa)))

    dk = (loss(k + eps, alpha) - loss(k - eps, alpha)) / (2.0 * eps)
    da = (loss(k, alpha + eps) - loss(k, alpha - eps)) / (2.0 * eps)
    return dk, da


def dftopk(r, k: int, alpha: float):
    """DFTopK, the comparator of §2 and of the supplement's "Comparison with
    DFTopK": a fixed threshold at the midpoint c = (r_(k) + r_(k+1))/2 of the
    k-th and (k+1)-th largest scores (integer k, 1 <= k < n; equal scores
    ranked by index as in `desc_order`) and a smooth step around it,
    p_i = 1 / (1 + exp(-(r_i - c)/t)).  Reading: the paper calls the step
    smooth without naming it; Table budget's relative mass error of 2.46 at
    alpha = -1, k = n/16 on Gaussian scores is what the logistic step gives
    (the Laplace CDF of Eq. (3) would give 1.65).
    Returns (p, c, (index of r_(k), index of r_(k+1)))."""
    r32 = np.asarray(r, dtype=np.float32).ravel()
    n = r32.size
    k = int(k)
    if not 1 <= k < n:
        raise ValueError("need an integer 1 <= k < n")
    t = -float(alpha)
    if not t > 0.0:
        raise ValueError("alpha must be negative")
    order = desc_order(r32)
    ik, ik1 = int(order[k - 1]), int(order[k])
    c = 0.5 * (float(r32[ik]) + float(r32[ik1]))
    u = (r32.astype(F64) - c) / t
    p = 1.0 / (1.0 + np.exp(-u))
    return p, c, (ik, ik1)


def dftopk_vjp(r, k: int, alpha: float, g) -> np.ndarray:
    """(grad_r p)^T g for `dftopk`: with s_i = p_i (1 - p_i) the logistic
    slope, dp_i/dr_j = (s_i/t)(delta_ij - dc/dr_j) and dc/dr_j = 1/2 for the
    two boundary scores only, so grad_j = g_j s_j / t minus
    (1/(2t)) sum_i g_i s_i at those two scores."""
    p, c, (ik, ik1) = dftopk(r, k, alpha)
    t = -float(alpha)
    g = _as_f64(g)
    s = p * (1.0 - p)
    out = g * s / t
    corr = math.fsum(g * s) / (2.0 * t)
    out[ik] -= corr
    out[ik1] -= corr
    return out


def budget_error(p, k: float) -> float:
    """|sum p - k|, with the sum of (possibly float32) p taken in float64."""
    return abs(math.fsum(np.asarray(p, dtype=F64).ravel()) - k)


def zero_temperature_threshold(r, k: int) -> float:
    """Theorem 1: as t -> 0 (distinct scores, integer k) the threshold tends to
    the midpoint of the k-th and (k+1)-th largest scores."""
    s = np.sort(_as_f64(r))[::-1]
    return 0.5 * (s[k - 1] + s[k])


# --------------------------------------------------------------------------
# Probabilistic bracket (§4, Suppl. B, Suppl. C)
# --------------------------------------------------------------------------

def bracket_ranks(n: int, k: float, K: int, z: float):
    """Eq. (8): 1-based ranks of the two order statistics.

    q = (n - k)/n, j = floor(Kq - z sqrt(Kq(1-q))), l = ceil(Kq + z sqrt(Kq(1-q))),
    evaluated left to right in IEEE float64 (Python floats never fuse a
    multiply-add).
    """
    q = (n - k) / n
    sd = math.sqrt(K * q * (1.0 - q))
    j = math.floor(K * q - z * sd)
    l = math.ceil(K * q + z * sd)
    return int(j), int(l), q


def splitmix64(seed: int, count: int) -> list[int]:
    """The first `count` outputs of SplitMix64 from state `seed` (Steele, Lea
    and Flood, "Fast splittable pseudorandom number generators", OOPSLA
    2014): the state advances by the golden-ratio increment 0x9E3779B97F4A7C15
    and each output is the state passed through the variant-13 mixing
    function (xor-shift 30, multiply 0xBF58476D1CE4E5B9, xor-shift 27,
    multiply 0x94D049BB133111EB, xor-shift 31), all modulo 2^64.  Python
    integers, one output at a time."""
    mask = (1 << 64) - 1
    state = seed & mask
    out = []
    for _ in range(count):
        state = (state + 0x9E3779B97F4A7C15) & mask
        x = state
        x = ((x ^ (x >> 30)) * 0xBF58476D1CE4E5B9) & mask
        x = ((x ^ (x >> 27)) * 0x94D049BB133111EB) & mask
        out.append(x ^ (x >> 31))
    return out


def counter_laplace_noise(seed: int, K: int, t: float) -> np.ndarray:
    """The library's default kernel noise for the bracket's sample (§4: a
    cached table of Laplace kernel noise; here drawn from a seed): draw s is
    the (s+1)-th SplitMix64 output z of `seed`, u = (2 floor(z / 2^12) + 1)
    / 2^53 (uniform, strictly inside (0, 1)), and the Laplace(0, t) inverse
    CDF of u, t ln(2u) below 1/2 and -t ln(2(1 - u)) above, in float64,
    rounded to float32."""
    z = splitmix64(seed, K)
    out = np.empty(K, dtype=np.float32)
    for s, v in enumerate(z):
        u = (2 * (v >> 12) + 1) / float(1 << 53)
        e = t * math.log(2.0 * u) if u < 0.5 else -t * math.log(2.0 * (1.0 - u))
        out[s] = np.float32(e)
    return out


def systematic_sample(r32, noise32) -> np.ndarray:
    """The deployed sampler of §4 (Suppl. C remark (iii)): a strided view of
    the scores plus a cached table of kernel noise,
    y_s = fl32(r[s * floor(n/K)] + eps_s), s = 0..K-1, added in float32."""
    r32 = np.asarray(r32, dtype=np.float32).ravel()
    eps = np.asarray(noise32, dtype=np.float32).ravel()
    K = eps.size
    stride = r32.size // K
    idx = np.arange(K, dtype=np.int64) * stride
    return (r32[idx] + eps).astype(np.float32)


def iid_sample(r32, idx, noise32) -> np.ndarray:
    """The sampler the coverage theorem assumes (Suppl. C, Theorem 2): K
    scores drawn uniformly with replacement, at indices idx that the caller
    draws, plus the kernel noise, y_s = fl32(r[idx_s] + eps_s)."""
    r32 = np.asarray(r32, dtype=np.float32).ravel()
    eps = np.asarray(noise32, dtype=np.float32).ravel()
    idx = np.asarray(idx, dtype=np.int64).ravel()
    if idx.size != eps.size or np.any(idx < 0) or np.any(idx >= r32.size):
        raise ValueError("need one index in [0, n) per noise draw")
    return (r32[idx] + eps).astype(np.float32)


def order_statistic(y32, j: int) -> float:
    """y_(j), the j-th smallest (1-based); -inf below 1 and +inf above K."""
    K = y32.size
    if j < 1:
        return -math.inf
    if j > K:
        return math.inf
    return float(np.sort(np.asarray(y32, dtype=np.float32))[j - 1])


@dataclasses.dataclass
class Partition:
    a_L: float
    a_R: float
    n_L: int
    n_M: int
    n_R: int
    T_L: float
    T_R: float
    m_idx: np.ndarray   # original indices of M in ascending index order


def partition(r32, a_L: float, a_R: float, t: float) -> Partition:
    """Suppl. B: L = {r < a_L}, M = {a_L <= r < a_R}, R = {r >= a_R} (float32
    comparisons), and the tail sums of Eq. (7),
        S_L = sum_{r < a_L} e^{(a_L - r)/alpha} = sum_L e^{-(a_L - r)/t},
        S_R = sum_{r >= a_R} e^{(r - a_R)/alpha} = sum_R e^{-(r - a_R)/t},
    every exponent <= 0, accumulated in float64."""
    r32 = np.asarray(r32, dtype=np.float32).ravel()
    aL32 = np.float32(a_L)
    aR32 = np.float32(a_R)
    inL = r32 < aL32
    inR = r32 >= aR32
    inM = ~(inL | inR)
    r = r32.astype(F64)
    T_L = math.fsum(np.exp(-(float(aL32) - r[inL]) / t)) if inL.any() else 0.0
    T_R = math.fsum(np.exp(-(r[inR] - float(aR32)) / t)) if inR.any() else 0.0
    return Partition(float(aL32), float(aR32), int(inL.sum()), int(inM.sum()),
                     int(inR.sum()), T_L, T_R, np.nonzero(inM)[0])


def solve_in_bracket(r32, part: Partition, k: float, t: float):
    """Suppl. B: exact root using only the sorted middle set and the tails.

    The R tail enters the prefix scan as a carry anchored at a_R, the L tail
    the suffix scan as a carry anchored at a_L; node values on the sorted M
    then equal LapSum at those scores, and the boundary cases (b above all of
    M, below all of M, M empty) are the same two-exponential equation.
    Returns (b, sorted M indices)."""
    r32 = np.asarray(r32, dtype=np.float32).ravel()
    midx = part.m_idx
    order = np.argsort(desc_keys(r32[midx]), kind="stable")
    m_sorted = midx[order]
    s = r32[m_sorted].astype(F64)
    above = (part.a_R, part.T_R) if part.n_R > 0 else None
    below = (part.a_L, part.T_L) if part.n_L > 0 else None
    b = _solve_on_sorted(s, k, t, part.n_R, above, below)
    return b, m_sorted


def widen(a_L: float, a_R: float, side: str):
    """One-sided doubling (Suppl. C, Expected Linear Runtime).

    side == "right" (LapSum(a_R) > k, so b >= a_R):
        a_L <- a_R,  a_R <- a_R + 2 (a_R - a_L)
    side == "left"  (LapSum(a_L) < k, so b < a_L):
        a_R <- a_L,  a_L <- a_L - 2 (a_R - a_L)
    Reading: both assignments use the old values; the arithmetic is float64
    on the float32 endpoints and the results are rounded to float32.
    """
    aL = float(np.float32(a_L))
    aR = float(np.float32(a_R))
    with np.errstate(invalid="ignore", over="ignore"):
        if side == "right":
            w = aR - aL
            new = (aR, aR + 2.0 * w)
        else:
            w = aR - aL
            new = (aL - 2.0 * w, aL)
    return float(np.float32(new[0])), float(np.float32(new[1]))


@dataclasses.dataclass
class BracketInfo:
    a_L: float
    a_R: float
    j: int
    l: int
    n_L: int
    n_M: int
    n_R: int
    T_L: float
    T_R: float
    lap_aL: float
    lap_aR: float
    attempts: int
    fell_back: int
    m_overflow: int


def bracketed_forward(r32, k: float, alpha: float, noise32, z: float = 5.16,
                      m_capacity: int | None = None, max_attempts: int = 3,
                      sample_idx=None):
    """Algorithm 1 with the validated path (§4, Suppl. C, Suppl. D).

    1. K = len(noise) kernel-noised samples by the systematic sampler, or by
       the i.i.d. sampler at the indices sample_idx when they are given;
    2. ranks j, l of Eq. (8); a_L = y_(j), a_R = y_(l);
    3. one pass: tails, counts, the middle set M;
    4. when |M| exceeds m_capacity (no room to hold M; widening only grows
       it) stop and solve by the full sort; otherwise the certificate
       LapSum(a_R) <= k <= LapSum(a_L) (plain sums here); on failure widen
       the failing side (one-sided doubling) and go to 3; after
       `max_attempts` brackets solve by the full sort;
    5. exact solve on the sorted M with the tails (Suppl. B);
    6. p_i = sigma((b - r_i)/alpha).
    Returns (p, b, info, sorted M indices or None after a fallback).
    """
    r32 = np.asarray(r32, dtype=np.float32).ravel()
    r, t = _check(r32, k, alpha)
    n = r32.size
    eps = np.asarray(noise32, dtype=np.float32).ravel()
    K = eps.size
    if not (2 <= K <= n):
        raise ValueError("need 2 <= K <= n")
    if m_capacity is None:
        m_capacity = n
    j, l, _q = bracket_ranks(n, k, K, z)
    y = systematic_sample(r32, eps) if sample_idx is None else iid_sample(r32, sample_idx, eps)
    a_L = order_statistic(y, j)
    a_R = order_statistic(y, l)
    info = BracketInfo(a_L, a_R, j, l, 0, 0, 0, 0.0, 0.0, 0.0, 0.0, 0, 0, 0)
    for attempt in range(1, max_attempts + 1):
        part = partition(r32, a_L, a_R, t)
        info = BracketInfo(part.a_L, part.a_R, j, l, part.n_L, part.n_M, part.n_R,
                           part.T_L, part.T_R, math.nan, math.nan, attempt, 0, 0)
        if part.n_M > m_capacity:
            # the certificate is read off the scan of the gathered M; an
            # attempt whose M does not fit is not certified at all
            info.m_overflow = 1
            break
        lap_R = 0.0 if math.isinf(a_R) and a_R > 0 else lapsum(r, a_R, t)
        lap_L = float(n) if math.isinf(a_L) and a_L < 0 else lapsum(r, a_L, t)
        info.lap_aL, info.lap_aR = lap_L, lap_R
        if lap_R <= k <= lap_L:
            b, m_sorted = solve_in_bracket(r32, part, k, t)
            return probs(r, b, alpha), b, info, m_sorted
        if attempt == max_attempts:
            break
        a_L, a_R = widen(a_L, a_R, "right" if lap_R > k else "left")
    info.fell_back = 1
    b = solve_sorted_scan(r, k, alpha)
    return probs(r, b, alpha), b, info, None
