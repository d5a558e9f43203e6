"""The parity comparison rules themselves (CPU): a planted error must fail them."""
import numpy as np
import pytest

from parity import check_param, check_update, rel, teacher_update

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


def _first_adam_step(w0, g, hyper):
    return teacher_update(w0, np.zeros_like(w0), np.zeros_like(w0), 0, g, hyper)


def test_check_update_catches_a_wrong_move():
    """One Adam step: the moves must match the oracle's relative to the largest
    move (a check of the parameter values alone could not see an error of one
    step at this learning rate)."""
    rng = np.random.default_rng(4)
    w0 = rng.standard_normal(1000) * 0.05
    g = rng.standard_normal(1000)
    ref = _first_adam_step(w0, g, ADAM)
    r, n = check_update(ref, w0, ref, w0, ADAM, 1e-4)
    assert r == 0.0 and n == 0
    bad = ref.copy()
    bad[11] = w0[11] + (ref[11] - w0[11]) * 0.9      # a 10% wrong step ...
    check_param(bad, ref, ADAM, 1, 2e-2, None)         # ... passes the value check
    with pytest.raises(AssertionError):
        check_update(bad, w0, ref, w0, ADAM, 2e-2)     # but not the update check


def test_check_update_teacher_rule():
    """An element whose oracle gradient is within the measured gradient error of
    zero may step either way, but only as the update rule applied to the GPU's
    own gradient says; every other element follows the oracle."""
    rng = np.random.default_rng(3)
    w0 = rng.standard_normal(1000) * 1e-2
    g = rng.standard_normal(1000)
    g[7] = 1e-4                                        # near zero
    ref = _first_adam_step(w0, g, ADAM)
    g_gpu = g + 1e-3 * rng.standard_normal(1000)       # the GPU's gradient, with noise
    g_gpu[7] = -2e-4                                   # sign flipped on the near-zero one
    gpu = _first_adam_step(w0, g_gpu, ADAM)
    und = np.abs(g) <= 2 * np.abs(g_gpu - g).max()
    assert und[7] and und.sum() < 20
    teach = _first_adam_step(w0, g_gpu, ADAM)
    r, n = check_update(gpu, w0, ref, w0, ADAM, 2e-2, undetermined=und, teacher=teach)
    assert n == und.sum()
    with pytest.raises(AssertionError):                # without the mask element 7 fails
        check_update(gpu, w0, ref, w0, ADAM, 2e-2)
    off = gpu.copy()
    off[7] = w0[7] + 0.5 * (gpu[7] - w0[7])            # not the update of its own gradient
    with pytest.raises(AssertionError):
        check_update(off, w0, ref, w0, ADAM, 2e-2, undetermined=und, teacher=teach)
    big = int(np.argmax(np.abs(g)))
    flip = _first_adam_step(w0, np.where(np.arange(1000) == big, -g_gpu, g_gpu), ADAM)
    with pytest.raises(AssertionError):                # a clear gradient fixes the direction
        check_update(flip, w0, ref, w0, ADAM, 2e-2, undetermined=und,
                     teacher=_first_adam_step(w0, np.where(np.arange(1000) == big, -g_gpu, g_gpu),
                                              ADAM))
    with pytest.raises(AssertionError):
        check_update(gpu, w0, ref, w0, ADAM, 2e-2, undetermined=und)   # mask needs a teacher


def test_check_update_eps_dominated_bound():
    rng = np.random.default_rng(5)
    w0 = rng.standard_normal(1000) * 1e-2
    g = rng.standard_normal(1000)
    ref = _first_adam_step(w0, g, ADAM)
    vh = np.abs(g)
    vh[3] = 1e-9                                       # eps-dominated by the oracle's record
    gpu = ref.copy()
    gpu[3] += 2 * ADAM["lr"]
    check_update(gpu, w0, ref, w0, ADAM, 1e-4, vh)
    gpu[3] += 10 * ADAM["lr"]                          # beyond Adam's largest move
    with pytest.raises(AssertionError):
        check_update(gpu, w0, ref, w0, ADAM, 1e-4, vh)


def test_undetermined_marks_sign_and_conditioning():
    """The oracle-decided set left to the teacher rule: on a first Adam step the
    elements whose gradient is within the measured error of zero (either sign
    is a valid outcome); on a later step the elements whose tiny gradient
    history makes m_hat / sqrt(v_hat) move by more than half the tolerance
    under that error; never a well-conditioned element or an exact zero."""
    from parity import undetermined
    n = 6
    w0 = np.full(n, 0.05)
    zeros = np.zeros(n)
    g = np.array([1.0, -0.5, 1e-9, 0.0, 0.3, 2.0])
    m_ref = (1 - ADAM["beta1"]) * g                 # first step from a zero state
    start = dict(params={"w": w0}, m={"w": zeros}, v={"w": zeros}, step={"w": 0})
    m_gpu = m_ref + np.array([1e-7, -1e-7, 0, 0, 0, 0])
    und = undetermined(m_gpu, m_ref, start, "w", ADAM, 1e-4)
    assert und.tolist() == [False, False, True, False, False, False]
    # step 2 from a history: element 2's history is ~1e-5, the others ~1
    m1 = np.array([0.1, -0.05, 1e-6, 0.03, 0.03, 0.2])
    v1 = np.array([1e-3, 2.5e-4, 1e-12, 9e-5, 9e-5, 4e-3])
    start2 = dict(params={"w": w0}, m={"w": m1}, v={"w": v1}, step={"w": 1})
    g2 = np.array([1.0, -0.5, 1e-5, 0.3, 0.3, 2.0])
    m_ref2 = ADAM["beta1"] * m1 + (1 - ADAM["beta1"]) * g2
    m_gpu2 = m_ref2 + 1e-7                          # a uniform measured error
    und2 = undetermined(m_gpu2, m_ref2, start2, "w", ADAM, 1e-4)
    assert und2[2] and not und2[[0, 1, 3, 4, 5]].any()
    assert not undetermined(m_ref2, m_ref2, start2, "w", ADAM, 1e-4).any()   # no error


def test_check_update_allows_the_weights_own_float32_rounding():
    """A float32 AdamW step on weights near 1 (LayerNorm scales) rounds the weight
    by up to ~1e-3 of a 1e-4 step; that much is allowed per element, more is not."""
    hyper = dict(kind="adamw", lr=1e-4, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01)
    rng = np.random.default_rng(9)
    w0 = 1.0 + rng.standard_normal(1000) * 0.01
    g = rng.standard_normal(1000)
    ref = teacher_update(w0, np.zeros(1000), np.zeros(1000), 0, g, hyper)
    w0f = np.asarray(w0, np.float32).astype(np.float64)
    gpu = np.asarray(ref, np.float32).astype(np.float64)     # the step rounded to float32
    check_update(gpu, w0f, ref, w0, hyper, 1e-4, teacher=ref)
    bad = gpu.copy()
    bad[4] += 5e-6                                            # 5% of a step: far beyond a rounding
    with pytest.raises(AssertionError):
        check_update(bad, w0f, ref, w0, hyper, 2e-2)


def test_teacher_rule_lifts_the_eps_dominated_cap_only():
    """Many eps-dominated elements fail the plain rules; with the teacher rule
    (which checks each of them exactly) they are accepted, and a wrong move on
    one of them is still caught."""
    rng = np.random.default_rng(12)
    w0 = rng.standard_normal(1000) * 0.05
    g = rng.standard_normal(1000)
    g[:50] = 1e-8 * rng.standard_normal(50)                # 5% eps-dominated
    ref = _first_adam_step(w0, g, ADAM)
    vh = np.abs(g)
    with pytest.raises(AssertionError):
        check_update(ref, w0, ref, w0, ADAM, 1e-4, vh)
    with pytest.raises(AssertionError):
        check_param(ref, ref, ADAM, 1, 1e-4, vh)
    check_update(ref, w0, ref, w0, ADAM, 1e-4, vh, teacher=ref)
    check_param(ref, ref, ADAM, 1, 1e-4, vh, covered=True)
    bad = ref.copy()
    bad[3] = w0[3] + 0.5 * (ref[3] - w0[3])
    with pytest.raises(AssertionError):
        check_update(bad, w0, ref, w0, ADAM, 1e-4, vh, teacher=ref)
