"""The parity comparison rules themselves (CPU): a planted error must fail them."""
import numpy as np
import pytest

from parity import check_param, rel

ADAM = dict(kind="adam", lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8)


def test_rel_is_max_norm_relative():
    assert rel([1.0, 2.0], [1.0, 2.0]) == 0.0
    assert rel([1.0, 2.5], [1.0, 2.0]) == pytest.approx(0.25)


def test_check_param_catches_a_wrong_well_conditioned_element():
    rng = np.random.default_rng(0)
    ref = rng.standard_normal(10000) * 0.05
    vh = np.full(10000, 1e-3)
    gpu = ref.copy()
    gpu[17] += 1e-4 * np.abs(ref).max() * 2
    with pytest.raises(AssertionError):
        check_param(gpu, ref, ADAM, 5, 1e-4, vh)


def test_check_param_bounds_eps_dominated_elements():
    rng = np.random.default_rng(1)
    ref = rng.standard_normal(10000) * 0.05
    vh = np.full(10000, 1e-3)
    vh[5] = 1e-9                               # eps-dominated by the oracle's own record
    gpu = ref.copy()
    gpu[5] += 3e-3                             # within 2 * K * 3.17 * lr for K = 5
    r, n = check_param(gpu, ref, ADAM, 5, 1e-4, vh)
    assert n == 1 and r == 0.0
    gpu[5] += 1.0                              # a garbage value still fails
    with pytest.raises(AssertionError):
        check_param(gpu, ref, ADAM, 5, 1e-4, vh)


def test_check_param_limits_the_excluded_fraction():
    ref = np.ones(1000)
    vh = np.full(1000, 1e-9)                   # everything eps-dominated: not acceptable
    with pytest.raises(AssertionError):
        check_param(ref, ref, ADAM, 5, 1e-4, vh)


def test_sgd_has_no_exclusions():
    ref = np.linspace(-1, 1, 100)
    gpu = ref.copy()
    gpu[3] += 1e-3
    with pytest.raises(AssertionError):
        check_param(gpu, ref, dict(kind="sgd", lr=0.1), 5, 1e-4, None)
