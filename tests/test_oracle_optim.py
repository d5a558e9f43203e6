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


# ---------------------------------------------------------------- Fig. 7's other optimizers
def test_adagrad_constant_gradient_closed_form():
    # With wd = 0 and a constant g the accumulated sum after s updates is s g^2, so
    # theta_t = theta_0 - eta * sum_{s=1..t} g / (sqrt(s) |g| + eps).
    g, eta, eps, T = np.array([0.5, -2.0, 1e-3]), 0.1, 1e-10, 7
    _, traj = _run("adagrad", [1.0, 1.0, 1.0], [g] * T, lr=eta, eps=eps, weight_decay=0.0)
    s = np.arange(1, T + 1)[:, None]
    want = 1.0 - eta * np.cumsum(g / (np.sqrt(s) * np.abs(g) + eps), axis=0)
    np.testing.assert_allclose(np.array(traj), want, rtol=1e-13, atol=1e-15)


@pytest.mark.parametrize("momentum", [0.0, 0.9])
def test_rmsprop_constant_gradient_closed_form(momentum):
    # With wd = 0 and a constant g: v_s = (1 - alpha^s) g^2, so each step's
    # normalised gradient is u_s = g / (sqrt(1 - alpha^s) |g| + eps); without
    # momentum theta moves by -eta u_s, with it by -eta sum_{r<=s} mu^(s-r) u_r.
    g, eta, alpha, eps, T = np.array([0.3, -4.0]), 0.01, 0.99, 1e-8, 6
    _, traj = _run("rmsprop", [0.0, 0.0], [g] * T, lr=eta, alpha=alpha, eps=eps,
                   momentum=momentum, weight_decay=0.0)
    s = np.arange(1, T + 1)[:, None]
    u = g / (np.sqrt(1.0 - alpha ** s) * np.abs(g) + eps)
    buf = np.array([sum(momentum ** (t - r) * u[r] for r in range(t + 1)) for t in range(T)])
    want = -eta * np.cumsum(buf if momentum else u, axis=0)
    np.testing.assert_allclose(np.array(traj), want, rtol=1e-12, atol=1e-15)


def test_adadelta_first_step_closed_form():
    # From m = v = 0: v_1 = (1 - rho) g^2 and d_1 = sqrt(eps / ((1 - rho) g^2 + eps)) g,
    # so with g^2 >> eps the first move is about sqrt(eps / (1 - rho)) sign(g).
    g, rho, eps, lr = np.array([2.0, -0.5, 0.0]), 0.9, 1e-6, 1.0
    p, traj = _run("adadelta", [0.0, 0.0, 0.0], [g], lr=lr, rho=rho, eps=eps, weight_decay=0.0)
    d1 = np.sqrt(eps / ((1.0 - rho) * g * g + eps)) * g
    np.testing.assert_allclose(traj[0], -lr * d1, rtol=1e-14, atol=0)
    np.testing.assert_allclose(p.m, (1.0 - rho) * d1 * d1, rtol=1e-14, atol=0)
    assert traj[0][2] == 0.0   # zero gradient: no move


@pytest.mark.parametrize("kind,hyper,torch_cls,torch_kw", [
    ("adagrad", dict(lr=0.05, eps=1e-10, weight_decay=1e-2), "Adagrad",
     dict(lr=0.05, eps=1e-10, weight_decay=1e-2)),
    ("rmsprop", dict(lr=0.01, alpha=0.99, eps=1e-8, weight_decay=1e-3, momentum=0.0), "RMSprop",
     dict(lr=0.01, alpha=0.99, eps=1e-8, weight_decay=1e-3)),
    ("rmsprop", dict(lr=0.01, alpha=0.9, eps=1e-8, weight_decay=1e-3, momentum=0.8), "RMSprop",
     dict(lr=0.01, alpha=0.9, eps=1e-8, weight_decay=1e-3, momentum=0.8)),
    ("adadelta", dict(lr=1.0, rho=0.9, eps=1e-6, weight_decay=1e-2), "Adadelta",
     dict(lr=1.0, rho=0.9, eps=1e-6, weight_decay=1e-2)),
])
def test_fig7_optimizers_match_torch_optim(kind, hyper, torch_cls, torch_kw):
    """The same published methods as implemented by torch.optim (float64, CPU),
    over random gradients with coupled weight decay."""
    import torch
    rng = np.random.default_rng(11)
    th0 = rng.standard_normal(64)
    gs = rng.standard_normal((8, 64))
    p, traj = _run(kind, th0, gs, **hyper)
    t = torch.tensor(th0, dtype=torch.float64, requires_grad=True)
    opt = getattr(torch.optim, torch_cls)([t], **torch_kw)
    for i, g in enumerate(gs):
        t.grad = torch.tensor(g, dtype=torch.float64)
        opt.step()
        np.testing.assert_allclose(traj[i], t.detach().numpy(), rtol=1e-12, atol=1e-14)


@pytest.mark.parametrize("kind,hyper", [
    ("sgd", dict(lr=0.1, momentum=0.9, weight_decay=1e-3)),
    ("adam", dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=1e-2)),
    ("adamw", dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=1e-2)),
    ("adagrad", dict(lr=1e-2, eps=1e-10, weight_decay=1e-4)),
    ("rmsprop", dict(lr=1e-2, alpha=0.99, eps=1e-8, weight_decay=1e-4, momentum=0.9)),
    ("adadelta", dict(lr=1.0, rho=0.9, eps=1e-6, weight_decay=1e-4)),
])
def test_sliced_application_equals_whole_tensor(kind, hyper):
    """apply() takes a tensor larger than SLICE slice by slice: bit-identical to
    the policy on the whole tensor (every policy is element-wise), including a
    ragged last slice and a non-contiguous 2-D input."""
    r = np.random.default_rng(5)
    n = 2 * optim.SLICE + 37
    theta, g = r.standard_normal(n), r.standard_normal(n)
    m, v = r.standard_normal(n) * 0.1, np.abs(r.standard_normal(n)) * 0.1
    policy = optim.POLICIES[kind]
    want = policy(theta, g, m, v, 3, **hyper)
    got = optim.apply_policy(policy, theta, g, m, v, 3, hyper)
    for a, b in zip(got, want):
        np.testing.assert_array_equal(a, b)
    # through apply() on a Param, from a transposed (non-contiguous) gradient
    rows = optim.SLICE // 512 + 3
    p = Param("w", theta[: rows * 512].reshape(rows, 512))
    p.m, p.v = m[: rows * 512].reshape(rows, 512), v[: rows * 512].reshape(rows, 512)
    p.step = 2
    gt = np.ascontiguousarray(g[: rows * 512].reshape(512, rows)).T
    p.grad = gt
    want = policy(p.value, gt, p.m, p.v, 3, **hyper)
    optim.apply(p, dict(hyper, kind=kind))
    for a, b in zip((p.value, p.m, p.v), want):
        np.testing.assert_array_equal(a, b)
