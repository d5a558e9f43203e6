"""Optimizer policies pi (Appendix A, Alg. 1: theta_t = theta_{t-1} + delta), float64.

`step` is the 1-based index t of the update being applied.

sgd   gradient descent with momentum (Appendix A, Eq. for pi_2):
          g' = g + wd * theta              (coupled weight decay; none in pi_2)
          b_t = alpha * b_{t-1} + g', b_0 = 0
          theta_t = theta_{t-1} - eta * b_t
      Unrolling b_t gives pi_2 = -eta * sum_tau alpha^(t-tau-1) g_tau exactly,
      and alpha = 0 gives plain gradient descent (pi_1).
adam  Adam (Kingma & Ba, Alg. 1; the optimizer of the paper's experimental
      settings), with coupled L2 weight decay g' = g + wd * theta:
          m_t = b1 m + (1 - b1) g'     v_t = b2 v + (1 - b2) g'^2
          theta_t = theta - (eta / (1 - b1^t)) * m_t / (sqrt(v_t) / sqrt(1 - b2^t) + eps)
adamw Adam with decoupled weight decay (Loshchilov & Hutter):
          theta <- theta * (1 - eta * wd), then the Adam step on the raw g.

Pinned by: closed forms on hand-set tensors (constant gradient) in
tests/test_oracle_optim.py.
"""
import numpy as np


def sgd(theta, g, m, v, step, lr, momentum, weight_decay, **_):
    g = g + weight_decay * theta
    m = momentum * m + g
    return theta - lr * m, m, v


def adam(theta, g, m, v, step, lr, beta1, beta2, eps, weight_decay=0.0, **_):
    g = g + weight_decay * theta
    m = beta1 * m + (1.0 - beta1) * g
    v = beta2 * v + (1.0 - beta2) * g * g
    bc1 = 1.0 - beta1 ** step
    bc2 = 1.0 - beta2 ** step
    return theta - (lr / bc1) * m / (np.sqrt(v) / np.sqrt(bc2) + eps), m, v


def adamw(theta, g, m, v, step, lr, beta1, beta2, eps, weight_decay, **_):
    theta = theta * (1.0 - lr * weight_decay)
    return adam(theta, g, m, v, step, lr, beta1, beta2, eps, 0.0)


POLICIES = {"sgd": sgd, "adam": adam, "adamw": adamw}


def apply(param, hyper):
    """Execute the optimizer of one parameter: consume its accumulated gradient.

    Reads and resets the gradient (Section 3, "read and reset by the optimizer"),
    updates the value and history, and counts the update.
    """
    policy = POLICIES[hyper["kind"]]
    step = param.step + 1
    param.value, param.m, param.v = policy(param.value, param.grad, param.m, param.v, step, **hyper)
    param.last_grad = param.grad   # kept for state snapshots only
    param.grad = None
    param.step = step
