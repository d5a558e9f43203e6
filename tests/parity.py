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
"""
import numpy as np

EPS_FACTOR = 100.0
MAX_SENSITIVE_FRACTION = 1e-2
MAX_UNDETERMINED_FRACTION = 0.75


def rel(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    den = np.max(np.abs(b)) if b.size else 0.0
    return float(np.max(np.abs(a - b)) / (den if den > 0 else 1.0)) if b.size else 0.0


def check_param(gpu, ref, hyper, steps, tol, min_sqrt_vhat=None, what="", ref_m=None,
                grad_tol=None):
    """Assert parity of one trained parameter tensor; returns (rel error, #sensitive).

    ref_m, grad_tol (one Adam step, optional): the oracle's first moment and the
    tolerance the test holds the moment itself to.  After one step Adam moves
    an element by lr * g / (|g| + eps), about lr * sign(g).  Where the oracle's
    |g| is within grad_tol * max|g| of zero, a run that meets the gradient
    tolerance may hold a gradient of either sign or of a size comparable with
    eps, and every move within Adam's bound is then a valid outcome; those
    elements (decided by the oracle) are held to that bound, at most
    MAX_UNDETERMINED_FRACTION of the tensor, and every other element to the
    tolerance.  This matters for bf16 operands, whose gradients carry ~1e-3
    relative noise.
    """
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    den = max(float(np.max(np.abs(ref))), 1e-30)
    err = np.abs(gpu - ref)
    if hyper["kind"] == "sgd" or min_sqrt_vhat is None:
        r = float(err.max() / den)
        assert r <= tol, f"{what}: rel {r:.3e} > {tol}"
        return r, 0
    sens = np.asarray(min_sqrt_vhat) < EPS_FACTOR * hyper["eps"]
    frac = float(sens.mean())
    assert frac <= MAX_SENSITIVE_FRACTION, f"{what}: eps-dominated fraction {frac:.2e}"
    if ref_m is not None and grad_tol is not None:
        am = np.abs(np.asarray(ref_m, np.float64))
        # exact zeros (a structurally zero gradient, e.g. the unused Q and K
        # thirds of a fused QKV weight) are exact on both sides
        und = (am <= grad_tol * am.max()) & (am > 0)
        uf = float(und.mean())
        assert uf <= MAX_UNDETERMINED_FRACTION, f"{what}: undetermined fraction {uf:.2e}"
        sens = sens | und
    r = float(err[~sens].max() / den) if (~sens).any() else 0.0
    assert r <= tol, f"{what}: rel {r:.3e} > {tol} on well-conditioned elements"
    if sens.any():
        step_bound = hyper["lr"] * (1 - hyper["beta1"]) / np.sqrt(1 - hyper["beta2"])
        bound = 2.0 * steps * step_bound + tol * den
        worst = float(err[sens].max())
        assert worst <= bound, f"{what}: sensitive element moved {worst:.3e} > {bound:.3e}"
    return r, int(sens.sum())


# A backward ReLU mask is a decision taken on a pre-activation; where that value
# lies within float32 rounding of 0 the GPU and the float64 oracle may decide
# differently, and one token's whole contribution then moves in every gradient
# below that layer (about 4 such decisions per step of the 8-layer width-1024
# MLP sit below one ulp of sum|w x|).  For layers under a ReLU the tests
# therefore bound the fraction of elements off by more than the tolerance and
# their distance (Adam's largest possible step), instead of the maximum.
MAX_TAINTED_FRACTION = 1e-2


def check_param_decisions(gpu, ref, hyper, steps, tol, what=""):
    """Parity of a parameter below a ReLU decision: returns (median rel, tainted fraction)."""
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    den = max(float(np.max(np.abs(ref))), 1e-30)
    err = np.abs(gpu - ref) / den
    frac = float((err > tol).mean())
    assert frac <= MAX_TAINTED_FRACTION, f"{what}: fraction {frac:.2e} off by more than {tol}"
    if hyper["kind"] == "sgd":
        bound = 2.0 * steps * hyper["lr"] * 10.0
    else:
        bound = 2.0 * steps * hyper["lr"] * (1 - hyper["beta1"]) / np.sqrt(1 - hyper["beta2"])
    assert float(err.max()) * den <= bound + tol * den, f"{what}: moved {err.max() * den:.3e}"
    return float(np.median(err)), frac
