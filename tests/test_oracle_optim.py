"""Pins for the oracle's optimizer policies: closed forms on hand-set tensors."""
import numpy as np
import pytest

from oracle import optim
from oracle.layers import Param


def _run(kind, theta0, grads, **hyper):
    p = Param("p", np.array(theta0, dtype=np.float64))
    traj = []
    for g in grads:
        p.grad = np.array(g, dtype=np.float64)
        optim.apply(p, dict(kind=kind, **hyper))
        traj.append(p.value.copy())
    return p, traj


def test_sgd_momentum_worked_values():
    # theta0 = 1, g = 0.5, lr = 0.1, momentum 0.9: b1 = 0.5, b2 = 0.95.
    _, traj = _run("sgd", [1.0], [[0.5]] * 2, lr=0.1, momentum=0.9, weight_decay=0.0)
    assert traj[0][0] == pytest.approx(0.95, abs=1e-15)
    assert traj[1][0] == pytest.approx(0.855, abs=1e-15)


def test_sgd_zero_momentum_is_gradient_descent():
    # Eq. for pi_1: delta = -eta * grad.
    rng = np.random.default_rng(0)
    th, g = rng.standard_normal(7), rng.standard_normal(7)
    _, traj = _run("sgd", th, [g], lr=0.3, momentum=0.0, weight_decay=0.0)
    np.testing.assert_allclose(traj[0], th - 0.3 * g, rtol=0, atol=1e-15)


def test_sgd_momentum_matches_pi2_sum():
    # Eq. for pi_2: delta_t = -eta * sum_{tau < t} alpha^(t - tau - 1) g_tau, summed over steps.
    rng = np.random.default_rng(3)
    eta, alpha, T = 0.05, 0.8, 9
    gs = rng.standard_normal((T, 5))
    th0 = rng.standard_normal(5)
    _, traj = _run("sgd", th0, gs, lr=eta, momentum=alpha, weight_decay=0.0)
    theta = th0.copy()
    for t in range(1, T + 1):
        delta = -eta * sum(alpha ** (t - tau - 1) * gs[tau] for tau in range(t))
        theta = theta + delta
        np.testing.assert_allclose(traj[t - 1], theta, rtol=1e-13, atol=1e-14)


def test_sgd_constant_gradient_closed_form():
    mu, lr, g, T = 0.9, 0.1, 0.5, 12
    _, traj = _run("sgd", [1.0], [[g]] * T, lr=lr, momentum=mu, weight_decay=0.0)
    for t in range(1, T + 1):
        expect = 1.0 - lr * g * sum((1 - mu ** s) / (1 - mu) for s in range(1, t + 1))
        assert traj[t - 1][0] == pytest.approx(expect, rel=1e-14)


def test_sgd_weight_decay_linear_recurrence():
    # g = 0: b_t = mu b_{t-1} + wd theta_{t-1} and theta_t = theta_{t-1} - lr b_t,
    # i.e. (theta, b) is multiplied by A = [[1 - lr wd, -lr mu], [wd, mu]] each step.
    lr, mu, wd, T = 0.1, 0.9, 0.05, 15
    A = np.array([[1 - lr * wd, -lr * mu], [wd, mu]])
    _, traj = _run("sgd", [2.0], [[0.0]] * T, lr=lr, momentum=mu, weight_decay=wd)
    for t in range(1, T + 1):
        expect = np.linalg.matrix_power(A, t) @ np.array([2.0, 0.0])
        assert traj[t - 1][0] == pytest.approx(expect[0], rel=1e-13)


@pytest.mark.parametrize("g", [0.5, -2.0, 1e-3])
def test_adam_constant_gradient(g):
    # Constant g: bias-corrected moments are g and g^2, so each step moves lr*g/(|g|+eps).
    lr, eps, T = 1e-3, 1e-8, 10
    p, traj = _run("adam", [0.3], [[g]] * T, lr=lr, beta1=0.9, beta2=0.999, eps=eps,
                   weight_decay=0.0)
    for t in range(1, T + 1):
        assert traj[t - 1][0] == pytest.approx(0.3 - t * lr * g / (abs(g) + eps), rel=1e-12)
    assert p.step == T
    assert p.m[0] == pytest.approx((1 - 0.9 ** T) * g, rel=1e-12)
    assert p.v[0] == pytest.approx((1 - 0.999 ** T) * g * g, rel=1e-12)


def test_adam_coupled_weight_decay_first_step():
    lr, wd, eps, th = 1e-2, 0.1, 1e-8, -0.7
    _, traj = _run("adam", [th], [[0.0]], lr=lr, beta1=0.9, beta2=0.999, eps=eps,
                   weight_decay=wd)
    gp = wd * th
    assert traj[0][0] == pytest.approx(th - lr * gp / (abs(gp) + eps), rel=1e-12)


def test_adamw_constant_gradient_geometric():
    lr, wd, eps, g, T, th0 = 1e-2, 0.1, 1e-8, 0.25, 20, 1.5
    _, traj = _run("adamw", [th0], [[g]] * T, lr=lr, beta1=0.9, beta2=0.999, eps=eps,
                   weight_decay=wd)
    c = 1 - lr * wd
    step = lr * g / (abs(g) + eps)
    for t in range(1, T + 1):
        expect = c ** t * th0 - step * (1 - c ** t) / (1 - c)
        assert traj[t - 1][0] == pytest.approx(expect, rel=1e-12)


def test_adam_zero_gradient_no_motion():
    _, traj = _run("adam", [0.4, -0.2], [[0.0, 0.0]] * 3, lr=1e-3, beta1=0.9, beta2=0.999,
                   eps=1e-8, weight_decay=0.0)
    np.testing.assert_array_equal(traj[-1], [0.4, -0.2])
