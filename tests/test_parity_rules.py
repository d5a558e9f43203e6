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


def test_check_param_undetermined_adam_step():
    """After one Adam step, an element whose oracle gradient is within the gradient
    tolerance of zero may move anywhere within Adam's bound; an element with a
    clear gradient may not, and nor may one beyond the bound."""
    rng = np.random.default_rng(3)
    ref = rng.standard_normal(1000) * 1e-3
    m = rng.standard_normal(1000)
    m[7] = 1e-4 * np.abs(m).max()            # within 2e-2 of zero
    vh = np.full(1000, 1.0)
    gpu = ref.copy()
    gpu[7] += 2 * ADAM["lr"]                  # the other direction
    r, n = check_param(gpu, ref, ADAM, 1, 2e-2, vh, ref_m=m, grad_tol=2e-2)
    assert n >= 1
    with pytest.raises(AssertionError):
        check_param(gpu, ref, ADAM, 1, 2e-2, vh)
    far = ref.copy()
    far[7] += 10 * ADAM["lr"]                 # beyond Adam's largest move
    with pytest.raises(AssertionError):
        check_param(far, ref, ADAM, 1, 2e-2, vh, ref_m=m, grad_tol=2e-2)
    big = int(np.argmax(np.abs(m)))
    bad = ref.copy()
    bad[big] += 2 * ADAM["lr"]
    with pytest.raises(AssertionError):       # a clear gradient fixes the step
        check_param(bad, ref, ADAM, 1, 2e-2, vh, ref_m=m, grad_tol=2e-2)
    flat = np.full(1000, 1e-6)
    flat[0] = 1.0
    with pytest.raises(AssertionError):       # nearly everything undetermined
        check_param(ref, ref, ADAM, 1, 2e-2, vh, ref_m=flat, grad_tol=2e-2)
