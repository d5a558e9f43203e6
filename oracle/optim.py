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

adagrad, rmsprop, adadelta  the other optimizers of the paper's comparison
      (Section 4, "Various Models and Optimizers", Fig. 7: SGD, SGD with
      momentum, Adagrad, RMSprop, Adam, Adadelta, weight decay applied unless
      stated).  The paper gives no formulas; these are the published methods
      (Duchi et al. 2011; Tieleman & Hinton's RMSprop; Zeiler 2012) in the form
      PyTorch implements them, with coupled weight decay g' = g + wd * theta:
      adagrad   v += g'^2;  theta -= eta * g' / (sqrt(v) + eps)
      rmsprop   v = alpha v + (1 - alpha) g'^2;  s = g' / (sqrt(v) + eps)
                momentum 0: theta -= eta * s;  else m = momentum m + s, theta -= eta * m
      adadelta  v = rho v + (1 - rho) g'^2;  d = sqrt(m + eps) / sqrt(v + eps) * g'
                m = rho m + (1 - rho) d^2;  theta -= eta * d
      (v: squared-gradient state, m: momentum buffer or squared-update state).

clip_scale  the global-norm clipping factor (forward-fusion's global-information
      step; see its docstring).

Pinned by: closed forms on hand-set tensors (constant gradient) in
tests/test_oracle_optim.py, where adagrad, rmsprop and adadelta are also run
against torch.optim's implementations in float64; clip_scale by a 3-4-5 closed form, the norm of the
concatenated gradients (numpy.linalg.norm) and the clipped norm in
tests/test_oracle_clip.py.
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


def adagrad(theta, g, m, v, step, lr, eps, weight_decay=0.0, **_):
    g = g + weight_decay * theta
    v = v + g * g
    return theta - lr * g / (np.sqrt(v) + eps), m, v


def rmsprop(theta, g, m, v, step, lr, alpha, eps, weight_decay=0.0, momentum=0.0, **_):
    g = g + weight_decay * theta
    v = alpha * v + (1.0 - alpha) * g * g
    s = g / (np.sqrt(v) + eps)
    if momentum != 0.0:
        m = momentum * m + s
        return theta - lr * m, m, v
    return theta - lr * s, m, v


def adadelta(theta, g, m, v, step, lr, rho, eps, weight_decay=0.0, **_):
    g = g + weight_decay * theta
    v = rho * v + (1.0 - rho) * g * g
    d = np.sqrt(m + eps) / np.sqrt(v + eps) * g
    m = rho * m + (1.0 - rho) * d * d
    return theta - lr * d, m, v


POLICIES = {"sgd": sgd, "adam": adam, "adamw": adamw, "adagrad": adagrad, "rmsprop": rmsprop,
            "adadelta": adadelta}


def clip_scale(grads, max_norm):
    """Factor for clipping gradients by their global norm, and that norm.

    Forward-fusion may change the gradients using information from every
    parameter before any of them is updated, and global-norm clipping is the
    example the paper gives (Appendix B.1; Table 1, "Global Info."); backward-
    fusion cannot, since it updates each tensor before the others' gradients
    exist (Section 3, "Backward-Fusion").  The paper names the operation
    without a formula; this takes the common definition:
        norm  = sqrt(sum over all gradient elements of g^2)
        scale = max_norm / (norm + 1e-6), capped at 1
    and every gradient is multiplied by scale before the optimizer uses it.
    A NaN norm gives a NaN scale (an infinite one gives 0).
    """
    total = 0.0
    for g in grads:
        total += float(np.sum(np.square(np.asarray(g, np.float64))))
    norm = float(np.sqrt(total))
    s = max_norm / (norm + 1e-6)
    return (1.0 if s > 1.0 else s), norm


# Elements per slice when a policy is applied to a large tensor (see apply).
SLICE = 1 << 20


def apply_policy(policy, theta, g, m, v, step, hyper):
    """policy(theta, g, m, v, step) over whole tensors.  Every policy above is
    element-wise (each output element depends on the same element of the inputs
    and on scalars only), so a large tensor is taken in slices of SLICE elements:
    the same operations on every element, with the temporaries small enough to
    stay in cache.  The result is identical to one call on the whole tensor."""
    if theta.size <= SLICE:
        return policy(theta, g, m, v, step, **hyper)
    outs = (np.empty_like(theta), np.empty_like(m), np.empty_like(v))
    flat_in = [np.ascontiguousarray(a).reshape(-1) for a in (theta, g, m, v)]
    flat_out = [o.reshape(-1) for o in outs]
    for s in range(0, theta.size, SLICE):
        sl = slice(s, s + SLICE)
        res = policy(*(a[sl] for a in flat_in), step, **hyper)
        for o, r in zip(flat_out, res):
            o[sl] = r
    return outs


def apply(param, hyper):
    """Execute the optimizer of one parameter: consume its accumulated gradient.

    Reads and resets the gradient (Section 3, "read and reset by the optimizer"),
    updates the value and history, and counts the update.
    """
    policy = POLICIES[hyper["kind"]]
    step = param.step + 1
    param.value, param.m, param.v = apply_policy(policy, param.value, param.grad, param.m,
                                                 param.v, step, hyper)
    param.last_grad = param.grad   # kept for state snapshots only
    param.grad = None
    param.step = step
