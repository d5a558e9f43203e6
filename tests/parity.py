"""Comparison rules shared by the GPU parity tests.

rel(a, b)    max-norm relative error ||a - b||_inf / ||b||_inf (b is the oracle).

Parameters trained by Adam / AdamW are compared element-class by element-class.
An element is eps-dominated when the oracle's bias-corrected sqrt(v_hat) fell
below EPS_FACTOR * eps at some step: there the update m_hat / (sqrt(v_hat) + eps)
has a derivative in the gradient of up to 1/eps, so the ~1e-9 float32 rounding
of a gradient contraction moves the element by a sizable fraction of a step in
ANY float32 implementation.  Which elements are eps-dominated is decided by the
oracle alone.  They must be a small fraction of the tensor and stay within the
largest distance two runs can drift apart, 2 * sum_t max|step_t|.  Adam's step
is at most lr * (1 - beta1) / sqrt(1 - beta2) per element (3.17 * lr for the
workloads' betas).  Every other element is held to the plain tolerance.

check_param compares parameter values, as the max relative error of the
metric is defined.  For one step of a small learning rate that is a weak
check (an AdamW step of lr 1e-4 moves a weight of magnitude ~0.08 by ~1e-4,
below 2e-2 of the weight's scale), so the one-step tests also compare the
update itself with check_update: the GPU's move from the state it started
from against the oracle's move, relative to the largest move.
"""
import numpy as np

EPS_FACTOR = 100.0
MAX_SENSITIVE_FRACTION = 1e-2
# Tolerance of the teacher-forced rule (an update recomputed from the GPU's own
# gradient), relative to the largest update.
TEACHER_TOL = 1e-3
# A float32 update step rounds the weight itself: the decay factor
# (1 - lr wd) is rounded to float32 (relative error <= 2^-24), then w * decay
# and w - step are each rounded (<= 2^-24 |w| each).  For a weight near 1 (a
# LayerNorm scale) that is ~1e-3 of an AdamW step of lr 1e-4, so each
# element's move may differ from the exact one by this much more.
F32_W_ROUNDING = 4.0 * 2.0 ** -24


def rel(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    den = np.max(np.abs(b)) if b.size else 0.0
    return float(np.max(np.abs(a - b)) / (den if den > 0 else 1.0)) if b.size else 0.0


def _adam_bound(hyper):
    return hyper["lr"] * (1 - hyper["beta1"]) / np.sqrt(1 - hyper["beta2"])


def check_param(gpu, ref, hyper, steps, tol, min_sqrt_vhat=None, what="", exclude=None,
                covered=False):
    """Assert parity of one trained parameter tensor; returns (rel error, #eps-dominated).

    exclude (bool mask, optional): elements left out of this rule because
    check_update's teacher rule checks them (the undetermined elements of a
    first Adam step; for a tensor that starts at zero, such as a bias, their
    value is the whole update and may take either sign).
    covered: the teacher rule checks every element of this step, so the
    eps-dominated elements need not be a small share of the tensor (their
    Adam bound here is loose; the teacher rule is not)."""
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    den = max(float(np.max(np.abs(ref))), 1e-30)
    err = np.abs(gpu - ref)
    if exclude is not None:
        err = np.where(np.asarray(exclude, bool), 0.0, err)
    if hyper["kind"] not in ("adam", "adamw") or min_sqrt_vhat is None:
        r = float(err.max() / den)
        assert r <= tol, f"{what}: rel {r:.3e} > {tol}"
        return r, 0
    sens = np.asarray(min_sqrt_vhat) < EPS_FACTOR * hyper["eps"]
    frac = float(sens.mean())
    assert covered or frac <= MAX_SENSITIVE_FRACTION, f"{what}: eps-dominated fraction {frac:.2e}"
    r = float(err[~sens].max() / den) if (~sens).any() else 0.0
    assert r <= tol, f"{what}: rel {r:.3e} > {tol} on well-conditioned elements"
    if sens.any():
        bound = 2.0 * steps * _adam_bound(hyper) + tol * den
        worst = float(err[sens].max())
        assert worst <= bound, f"{what}: sensitive element moved {worst:.3e} > {bound:.3e}"
    return r, int(sens.sum())


def check_update(gpu_new, gpu_start, ref_new, ref_start, hyper, tol, min_sqrt_vhat=None,
                 what="", undetermined=None, teacher=None):
    """Assert that one step moved a parameter tensor as the oracle's step did.

    The GPU's move gpu_new - gpu_start (gpu_start: the float32 values it started
    from) against the oracle's ref_new - ref_start, element by element, within
    tol of the oracle's largest move beyond the weight's own float32 rounding
    (F32_W_ROUNDING |w| per element).  Adam's eps-dominated elements (decided by
    the oracle's min_sqrt_vhat) are held to Adam's largest step instead.

    teacher (optional): the oracle's update formula applied to the GPU's own
    gradient, from gpu_start (the test reconstructs the gradient from the GPU's
    first moment).  When given, EVERY element's move must equal the teacher's
    within TEACHER_TOL of the oracle's largest move: the GPU applied the update
    rule correctly to the gradient it computed, and the separate comparison of
    that gradient (its first moment) with the oracle's checks the gradient.
    undetermined (bool mask, optional; only with teacher) marks elements whose
    update the oracle does not fix at the measured gradient error (see
    undetermined()); those are left out of the oracle rule and checked by the
    teacher rule alone.
    Returns (rel error on the oracle-checked elements, number of undetermined
    elements).
    """
    d_gpu = np.asarray(gpu_new, np.float64) - np.asarray(gpu_start, np.float64)
    d_ref = np.asarray(ref_new, np.float64) - np.asarray(ref_start, np.float64)
    den = max(float(np.max(np.abs(d_ref))), 1e-30)
    # errors beyond the weight's own float32 rounding, relative to the largest move
    slack = F32_W_ROUNDING * np.abs(np.asarray(gpu_start, np.float64))
    err = np.maximum(np.abs(d_gpu - d_ref) - slack, 0.0)
    held = np.zeros(d_ref.shape, bool)
    if teacher is not None:
        d_teach = np.asarray(teacher, np.float64) - np.asarray(gpu_start, np.float64)
        r_t = float(np.maximum(np.abs(d_gpu - d_teach) - slack, 0.0).max() / den)
        assert r_t <= TEACHER_TOL, f"{what}: move off the update of its own gradient by {r_t:.3e}"
    if hyper["kind"] in ("adam", "adamw") and min_sqrt_vhat is not None:
        sens = np.asarray(min_sqrt_vhat) < EPS_FACTOR * hyper["eps"]
        # with the teacher rule every element is checked exactly; without it the
        # elements held only to Adam's bound must be few
        assert teacher is not None or float(sens.mean()) <= MAX_SENSITIVE_FRACTION, \
            f"{what}: eps-dominated fraction {float(sens.mean()):.2e}"
        if sens.any():
            worst = float(err[sens].max())
            bound = 2.0 * _adam_bound(hyper) + tol * den
            assert worst <= bound, f"{what}: eps-dominated element moved {worst:.3e} > {bound:.3e}"
        held |= sens
    n_und = 0
    if undetermined is not None:
        assert teacher is not None, "undetermined elements need the teacher rule"
        und = np.asarray(undetermined, bool)
        n_und = int(und.sum())
        held |= und
    r = float(err[~held].max() / den) if (~held).any() else 0.0
    assert r <= tol, f"{what}: update rel {r:.3e} > {tol}"
    return r, n_und


def teacher_update(w_start, m_start, v_start, step_start, grad, hyper):
    """The oracle's update rule (float64) applied once to a given gradient."""
    from oracle import layers as OL, optim as OO
    p = OL.Param("teacher", np.asarray(w_start, np.float64))
    p.m = np.asarray(m_start, np.float64).copy()
    p.v = np.asarray(v_start, np.float64).copy()
    p.step = int(step_start)
    p.grad = np.asarray(grad, np.float64)
    OO.apply(p, hyper)
    return p.value


def _f32(a):
    return np.asarray(np.asarray(a, np.float32), np.float64)


def gpu_gradient(m_new, m_start, w_start, hyper):
    """The gradient a GPU step consumed, recovered from its first moment
    m_new = beta1 m_start + (1 - beta1) g' (g' = g + wd w for Adam's coupled decay)."""
    g = (np.asarray(m_new, np.float64) - hyper["beta1"] * np.asarray(m_start, np.float64)) \
        / (1.0 - hyper["beta1"])
    if hyper["kind"] == "adam":
        g = g - hyper.get("weight_decay", 0.0) * np.asarray(w_start, np.float64)
    return g


def teachers(st, start, hyper):
    """Per tensor: the oracle's update applied to the GPU's own gradient, from
    the float32 start state the GPU stepped from (Adam family only)."""
    if hyper["kind"] not in ("adam", "adamw"):
        return {}
    out = {}
    for k in st["params"]:
        w0, m0, v0 = _f32(start["params"][k]), _f32(start["m"][k]), _f32(start["v"][k])
        g = gpu_gradient(st["m"][k], m0, w0, hyper)
        out[k] = teacher_update(w0, m0, v0, start["step"][k], g, hyper)
    return out


def undetermined(m_gpu, m_ref, start, k, hyper, tol):
    """Elements of tensor k whose update the oracle does not fix at the
    measured gradient error: the oracle's update rule, applied from the step's
    start state to the oracle's gradient moved by +-delta (delta: the largest
    first-moment error of the tensor over (1 - beta1)), moves the element by
    more than half the tolerance of the largest update.  This takes in the
    sign of a first Adam step (an update of +-lr whatever the gradient's size)
    and, later, elements whose small gradient history makes m_hat / sqrt(v_hat)
    sensitive to the gradient's float32 rounding.  Exact zeros on both sides
    (a structurally zero gradient) are not counted."""
    m_gpu = np.asarray(m_gpu, np.float64)
    m_ref = np.asarray(m_ref, np.float64)
    w0, m0, v0, t0 = (np.asarray(start["params"][k], np.float64), np.asarray(start["m"][k], np.float64),
                      np.asarray(start["v"][k], np.float64), start["step"][k])
    delta = float(np.max(np.abs(m_gpu - m_ref))) / (1.0 - hyper["beta1"])
    g = gpu_gradient(m_ref, m0, w0, hyper)
    u = teacher_update(w0, m0, v0, t0, g, hyper)
    dev = np.maximum(np.abs(teacher_update(w0, m0, v0, t0, g + delta, hyper) - u),
                     np.abs(teacher_update(w0, m0, v0, t0, g - delta, hyper) - u))
    band = 0.5 * tol * float(np.max(np.abs(u - w0)))
    return (dev > band) & ~((m_ref == 0.0) & (m_gpu == 0.0))
