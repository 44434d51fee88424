"""Planted mistakes: each deliberately broken copy of an oracle routine must
fail at least one pin.  The mistakes are planted in the oracle, on the CPU,
through pytest's monkeypatch; nothing here touches the GPU library."""
import math

import numpy as np
import pytest

import oracle.lapsum_oracle as O
import pins

_F64 = np.float64


def _bad_cdf_sign(u):
    u = np.asarray(u, dtype=_F64)
    out = np.empty_like(u)
    neg = u <= 0.0
    out[neg] = 0.5 * np.exp(-u[neg])          # wrong exponent sign
    out[~neg] = 1.0 - 0.5 * np.exp(u[~neg])
    return out


def _bad_cdf_branch(u):
    u = np.asarray(u, dtype=_F64)
    out = np.empty_like(u)
    neg = u < -0.5                            # wrong branch point
    out[neg] = 0.5 * np.exp(u[neg])
    out[~neg] = 1.0 - 0.5 * np.exp(-u[~neg])
    return out


_orig_node_curve = O._node_curve
_orig_gap_root = O._gap_root
_orig_bracket_ranks = O.bracket_ranks
_orig_partition = O.partition
_orig_vjp = O.vjp
_orig_lapsum = O.lapsum
_orig_counter_noise = O.counter_laplace_noise
_orig_initial_bracket = O.initial_bracket


def _bad_node_full_E(s, t, n_above, above, below):
    logP, logQ, N = _orig_node_curve(s, t, n_above, above, below)
    i = np.arange(1, s.size + 1, dtype=_F64)
    E = 2.0 * (N - n_above - i + 0.5 * np.exp(logP))
    return logP, logQ, n_above + i - 0.5 * np.exp(logP) + E     # dropped the 1/2 on E


def _bad_node_inclusive_E(s, t, n_above, above, below):
    logP, logQ, N = _orig_node_curve(s, t, n_above, above, below)
    i = np.arange(1, s.size + 1, dtype=_F64)
    return logP, logQ, n_above + i - 0.5 * np.exp(logP) + 0.5 * np.exp(logQ)  # inclusive suffix


def _bad_node_rank(s, t, n_above, above, below):
    logP, logQ, N = _orig_node_curve(s, t, n_above, above, below)
    return logP, logQ, N - 1.0                # 0-based rank


def _bad_gap_sign(k, t, c_up, up, down):
    return _orig_gap_root(2.0 * c_up - k if up is not None and down is not None else k, t, c_up, up, down)


def _bad_brent_budget(r, k, alpha):
    from scipy.optimize import brentq
    t = -float(alpha)
    lo, hi = O.initial_bracket(r, k, t)
    n = np.asarray(r).size
    # root of LapSum(b) = n - k: the budget counted from the wrong end
    return float(brentq(lambda b: _orig_lapsum(r, b, t) - (n - k), lo - 50 * t, hi + 50 * t,
                        xtol=1e-14 * t))


def _bad_brent_tolerance(r, k, alpha):
    from scipy.optimize import brentq
    t = -float(alpha)
    lo, hi = O.initial_bracket(r, k, t)
    return float(brentq(lambda b: _orig_lapsum(r, b, t) - k, lo, hi, xtol=1e-3 * t))  # loose


def _bad_certify_swapped(r, k, alpha, b, delta):
    t = -float(alpha)
    return _orig_lapsum(r, b + delta, t) > k > _orig_lapsum(r, b - delta, t)   # wrong sides


def _bad_certify_one_sided(r, k, alpha, b, delta):
    t = -float(alpha)
    return _orig_lapsum(r, b - delta, t) > k                  # upper side never checked


def _bad_splitmix_shift(seed, count):
    mask = (1 << 64) - 1
    state, out = seed & mask, []
    for _ in range(count):
        state = (state + 0x9E3779B97F4A7C15) & mask
        x = state
        x = ((x ^ (x >> 31)) * 0xBF58476D1CE4E5B9) & mask     # 31 for 30
        x = ((x ^ (x >> 27)) * 0x94D049BB133111EB) & mask
        out.append(x ^ (x >> 31))
    return out


def _bad_noise_scale(seed, K, t):
    return _orig_counter_noise(seed, K, 2.0 * t)              # Laplace(0, 2t)


def _bad_noise_branch(seed, K, t):
    return -_orig_counter_noise(seed, K, t)                   # branches swapped


def _bad_vjp_unnormalised(r, b, alpha, g):
    t = -float(alpha)
    r = np.asarray(r, _F64).ravel()
    g = np.asarray(g, _F64).ravel()
    f = np.exp(-np.abs(b - r) / t) / (2.0 * t)
    return f * (g - math.fsum(g * f))         # q = f, not f / sum f


def _bad_vjp_scale(r, b, alpha, g):
    return 2.0 * _orig_vjp(r, b, alpha, g)    # f without the 1/(2t)... off by 2


def _params_sums(r, b, alpha, g):
    t = -float(alpha)
    r = np.asarray(r, _F64)
    g = np.asarray(g, _F64)
    u = (r - b) / t
    s = 0.5 * np.exp(-np.abs(u))
    return t, s.sum(), (s * g).sum(), (s * u).sum(), (s * g * u).sum()


def _bad_params_mean_sign(r, b, alpha, g):
    t, F, G, U, H = _params_sums(r, b, alpha, g)
    return G / F, (H + (U / F) * G) / t       # wrong sign of the centring term


def _bad_params_no_centre(r, b, alpha, g):
    t, F, G, U, H = _params_sums(r, b, alpha, g)
    return G / F, H / t                        # db/dalpha dropped


def _bad_params_t(r, b, alpha, g):
    t, F, G, U, H = _params_sums(r, b, alpha, g)
    return G / F, (H - (U / F) * G) / (t * t)  # u differentiated as r/t


def _bad_params_k_unnormalised(r, b, alpha, g):
    t, F, G, U, H = _params_sums(r, b, alpha, g)
    return G / t, (H - (U / F) * G) / t        # dp/dk taken as s/t


def _bad_ranks_sd(n, k, K, z):
    q = (n - k) / n
    sd = math.sqrt(K * q)                     # dropped (1 - q)
    return math.floor(K * q - z * sd), math.ceil(K * q + z * sd), q


def _bad_ranks_q(n, k, K, z):
    q = k / n                                 # transposed quantile
    sd = math.sqrt(K * q * (1.0 - q))
    return math.floor(K * q - z * sd), math.ceil(K * q + z * sd), q


def _bad_partition_closed(r32, a_L, a_R, t):
    r32 = np.asarray(r32, np.float32).ravel()
    p = _orig_partition(r32, a_L, a_R, t)
    inL = r32 <= np.float32(a_L)              # wrong boundary side
    p.n_L = int(inL.sum())
    p.m_idx = np.nonzero(~inL & (r32 < np.float32(a_R)))[0]
    p.n_M = int(p.m_idx.size)
    return p


def _bad_partition_tail_sign(r32, a_L, a_R, t):
    p = _orig_partition(r32, a_L, a_R, t)
    r = np.asarray(r32, np.float32).ravel().astype(_F64)
    inR = r >= np.float32(a_R)
    p.T_R = math.fsum(np.exp(-(r[inR] - a_R) / t) * 0.5)  # halved tail
    return p


def _bad_widen(a_L, a_R, side):
    aL, aR = float(np.float32(a_L)), float(np.float32(a_R))
    if side == "right":
        aL = aR
        aR = aR + 2.0 * (aR - aL)             # uses the updated a_L
    else:
        aR = aL
        aL = aL - 2.0 * (aR - aL)
    return float(np.float32(aL)), float(np.float32(aR))


def _bad_order_stat(y32, j):
    K = y32.size
    if j < 0:
        return -math.inf
    if j >= K:
        return math.inf
    return float(np.sort(np.asarray(y32, np.float32))[j])   # 0-based


def _bad_sampler(r32, noise32):
    r32 = np.asarray(r32, np.float32).ravel()
    eps = np.asarray(noise32, np.float32).ravel()
    stride = -(-r32.size // eps.size)         # ceil instead of floor
    idx = np.minimum(np.arange(eps.size) * stride, r32.size - 1)
    return (r32[idx] + eps).astype(np.float32)


def _bad_iid_sample(r32, idx, noise32):
    return O.systematic_sample(r32, noise32)  # the indices ignored


_orig_dftopk = O.dftopk
_orig_dftopk_vjp = O.dftopk_vjp


def _bad_dftopk_step(r, k, alpha):
    p, c, b = _orig_dftopk(r, k, alpha)
    u = (np.asarray(r, np.float32).astype(_F64) - c) / -alpha
    return np.where(u <= 0, 0.5 * np.exp(u), 1 - 0.5 * np.exp(-u)), c, b   # Laplace CDF step


def _bad_dftopk_ranks(r, k, alpha):
    r32 = np.asarray(r, np.float32).ravel()
    o = O.desc_order(r32)
    p, _, _ = _orig_dftopk(r, k, alpha)
    c = 0.5 * (float(r32[o[k - 1]]) + float(r32[o[max(k - 2, 0)]]))   # r_(k-1), r_(k)
    u = (r32.astype(_F64) - c) / -alpha
    return 1.0 / (1.0 + np.exp(-u)), c, (int(o[k - 1]), int(o[max(k - 2, 0)]))


def _bad_dftopk_vjp(r, k, alpha, g):
    p = _orig_dftopk(r, k, alpha)[0]
    return np.asarray(g, _F64) * p * (1 - p) / -alpha   # threshold held fixed


MUTANTS = {
    "cdf_sign": ("laplace_cdf", _bad_cdf_sign),
    "cdf_branch": ("laplace_cdf", _bad_cdf_branch),
    "node_E_half_dropped": ("_node_curve", _bad_node_full_E),
    "node_E_inclusive": ("_node_curve", _bad_node_inclusive_E),
    "node_rank_off_by_one": ("_node_curve", _bad_node_rank),
    "gap_root_sign": ("_gap_root", _bad_gap_sign),
    "brent_budget_from_wrong_end": ("solve_brent", _bad_brent_budget),
    "brent_loose_tolerance": ("solve_brent", _bad_brent_tolerance),
    "certify_swapped_sides": ("certify_root", _bad_certify_swapped),
    "certify_one_sided": ("certify_root", _bad_certify_one_sided),
    "splitmix_shift": ("splitmix64", _bad_splitmix_shift),
    "noise_scale": ("counter_laplace_noise", _bad_noise_scale),
    "noise_branch": ("counter_laplace_noise", _bad_noise_branch),
    "vjp_unnormalised_q": ("vjp", _bad_vjp_unnormalised),
    "vjp_scale": ("vjp", _bad_vjp_scale),
    "params_mean_sign": ("vjp_params", _bad_params_mean_sign),
    "params_no_centre": ("vjp_params", _bad_params_no_centre),
    "params_t": ("vjp_params", _bad_params_t),
    "params_k_unnormalised": ("vjp_params", _bad_params_k_unnormalised),
    "ranks_sd": ("bracket_ranks", _bad_ranks_sd),
    "ranks_q": ("bracket_ranks", _bad_ranks_q),
    "partition_boundary": ("partition", _bad_partition_closed),
    "partition_tail": ("partition", _bad_partition_tail_sign),
    "widen_sequential": ("widen", _bad_widen),
    "order_stat_0based": ("order_statistic", _bad_order_stat),
    "sampler_stride": ("systematic_sample", _bad_sampler),
    "iid_sampler_ignores_indices": ("iid_sample", _bad_iid_sample),
    "dftopk_laplace_step": ("dftopk", _bad_dftopk_step),
    "dftopk_wrong_pair": ("dftopk", _bad_dftopk_ranks),
    "dftopk_vjp_fixed_threshold": ("dftopk_vjp", _bad_dftopk_vjp),
}

CHECKS = [
    pins.check_n1_closed_form, pins.check_all_equal_closed_form,
    pins.check_symmetric_half_budget, pins.check_invariants,
    lambda: pins.check_bisect_matches_scan(6),
    pins.check_decimal_bruteforce,
    lambda: pins.check_brent(4), pins.check_certify_root,
    lambda: pins.check_splitmix64([(1234567, (6457827717110365317, 3203168211198807973))]),
    pins.check_counter_noise,
    lambda: pins.check_vjp_fd(((1, 16, 4, -1.0),), tol=1e-8),
    pins.check_vjp_invariants,
    lambda: pins.check_params_fd(((24, 6.0, -1.0), (40, 13.5, -0.3)), tol=1e-6),
    pins.check_params_closed_forms, pins.check_params_scale_identity,
    pins.check_dftopk_fd, pins.check_dftopk_midpoint_is_the_zero_temperature_threshold,
    lambda: pins.check_dftopk_budget_table([(10000, 2.46), (100000, 2.47)]),
    pins.check_bracket_ranks, pins.check_partition_definition,
    pins.check_sampler_and_order_statistic, pins.check_widen_rule,
    pins.check_bracket_equals_full, pins.check_forced_widening,
]


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(name, monkeypatch):
    attr, bad = MUTANTS[name]
    monkeypatch.setattr(O, attr, bad)
    failed = []
    for chk in CHECKS:
        try:
            with np.errstate(all="ignore"):
                chk()
        except (AssertionError, ValueError, ZeroDivisionError, IndexError, FloatingPointError):
            failed.append(getattr(chk, "__name__", "lambda"))
            break
    assert failed, f"mutant {name} passed every pin"


def test_unmutated_oracle_passes_the_same_checks():
    for chk in CHECKS:
        chk()
