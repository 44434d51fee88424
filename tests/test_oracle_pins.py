"""The float64 oracle pinned against closed forms, invariants, high-precision
brute force, finite differences and the bracket theorem (CPU only)."""
import os

import numpy as np
import pytest

import oracle.lapsum_oracle as O
import pins

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_bisection_matches_sorted_scan():
    pins.check_bisect_matches_scan()


def test_single_score_closed_form():
    pins.check_n1_closed_form()


def test_all_equal_scores_closed_form():
    pins.check_all_equal_closed_form()


def test_symmetric_scores_half_budget_threshold_is_zero():
    pins.check_symmetric_half_budget()


def test_zero_temperature_limit_is_midpoint():
    pins.check_zero_temperature()


def test_shift_scale_permutation_equivariance():
    pins.check_equivariance()


def test_output_invariants():
    pins.check_invariants()


def test_decimal_bruteforce_tiny():
    pins.check_decimal_bruteforce()


def test_brent_matches_bisection_and_closed_form():
    pins.check_brent()


def test_certificate_at_known_roots():
    pins.check_certify_root()


def _gradcheck_rows():
    rows, thr = [], None
    with open(os.path.join(GOLDEN, "gradcheck_table.txt")) as fh:
        for line in fh:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            parts = line.split()
            if parts[0] == "pass_threshold":
                thr = float(parts[1])
            else:
                rows.append((int(parts[0]), int(parts[1]), float(parts[2]), float(parts[3])))
    return rows, thr


def test_vjp_matches_finite_differences_on_paper_configs():
    rows, thr = _gradcheck_rows()
    assert len(rows) == 3 and thr == 1e-3
    worst = pins.check_vjp_fd(tuple(rows), tol=1e-8)
    assert worst < thr


def test_vjp_invariants():
    pins.check_vjp_invariants()


def test_budget_and_temperature_gradients_match_finite_differences():
    worst = pins.check_params_fd()
    assert worst < 1e-6


def test_budget_and_temperature_gradients_closed_forms():
    pins.check_params_closed_forms()


def test_temperature_gradient_scale_identity():
    pins.check_params_scale_identity()


def test_descending_order_and_ties():
    pins.check_desc_order()


def test_bracket_ranks_cover_binomial_quantile():
    pins.check_bracket_ranks()
    j, l, _ = O.bracket_ranks(10**7, 2000.0, 46416, 5.16)
    assert l > 46416            # a_R = +inf for the n = 1e7 workload
    j, l, _ = O.bracket_ranks(10**8, 20000.0, 10**5, 5.16)
    assert l > 10**5


def test_partition_sets_and_tails():
    pins.check_partition_definition()


def test_bracketed_solve_equals_definition():
    pins.check_bracket_equals_full()


def test_forced_misses_widen_and_stay_exact():
    pins.check_forced_widening()


def test_sampler_and_order_statistic():
    pins.check_sampler_and_order_statistic()


def test_widening_rule():
    pins.check_widen_rule()


def test_iid_bracket_coverage_matches_binomial():
    pins.check_coverage_theorem()


def _budget_rows():
    out = []
    with open(os.path.join(GOLDEN, "budget_table.txt")) as fh:
        for line in fh:
            if line.strip() and not line.startswith("#"):
                n, bound = line.split()
                out.append((int(n), float(bound)))
    return out


def test_budget_accuracy_table():
    rows = _budget_rows()
    assert all(b == 1e-5 for _, b in rows)
    pins.check_budget_table(tuple(n for n, _ in rows if n <= 100000))


def test_oracle_rejects_invalid_arguments():
    x = np.zeros(4, dtype=np.float32)
    for k, a in ((0.0, -1.0), (4.0, -1.0), (1.0, 0.0), (1.0, 1.0), (float("nan"), -1.0)):
        with pytest.raises(ValueError):
            O.solve_bisect(x, k, a)
    with pytest.raises(ValueError):
        O.solve_bisect(np.array([np.inf], dtype=np.float32), 0.5, -1.0)


def _dftopk_rows():
    rows = []
    with open(os.path.join(GOLDEN, "dftopk_budget_table.txt")) as fh:
        for line in fh:
            line = line.strip()
            if line and not line.startswith("#"):
                n, v = line.split()
                rows.append((int(n), float(v)))
    return rows


def test_dftopk_budget_error_matches_the_table():
    rows = _dftopk_rows()
    assert [n for n, _ in rows] == [1000, 10000, 100000, 1000000, 10000000]
    pins.check_dftopk_budget_table([r for r in rows if r[0] <= 1000000])


def test_dftopk_vjp_matches_finite_differences():
    pins.check_dftopk_fd()


def test_dftopk_midpoint_is_the_zero_temperature_threshold():
    pins.check_dftopk_midpoint_is_the_zero_temperature_threshold()


def _splitmix_rows():
    rows = []
    with open(os.path.join(GOLDEN, "splitmix64_vectors.txt")) as fh:
        for line in fh:
            line = line.strip()
            if line and not line.startswith("#"):
                v = [int(x) for x in line.split()]
                rows.append((v[0], tuple(v[1:])))
    return rows


def test_splitmix64_published_outputs():
    rows = _splitmix_rows()
    assert rows and len(rows[0][1]) == 5
    pins.check_splitmix64(rows)


def test_counter_noise_is_laplace():
    pins.check_counter_noise()
