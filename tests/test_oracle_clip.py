"""Pins for the oracle's global-norm gradient clipping (forward-fusion's
global-information step, Appendix B.1 and Table 1).

The factor is pinned by a closed form (a 3-4-5 triangle), by numpy's norm of
the concatenated gradients and by the norm of the clipped gradients.  The
training path is pinned by the first SGD step written out by hand from the
unclipped gradient, by the ordering invariant (eager and forward-fusion clip
the same gradients at the same point, so they stay bit-identical) and by
backward-fusion refusing the option.
"""
import math

import numpy as np
import pytest

from oracle import run
from oracle.optim import clip_scale
from workloads import get_config, reduced_config


def test_clip_scale_closed_form():
    scale, norm = clip_scale([np.array([3.0]), np.array([[4.0]])], 1.0)
    assert norm == 5.0
    assert scale == 1.0 / (5.0 + 1e-6)
    scale, norm = clip_scale([np.array([3.0, 4.0])], 10.0)
    assert (scale, norm) == (1.0, 5.0)


def test_clip_scale_is_the_norm_of_the_concatenation():
    r = np.random.default_rng(3)
    gs = [r.standard_normal(s) for s in [(7, 5), (5,), (3, 4, 2), (1,)]]
    scale, norm = clip_scale(gs, 0.5)
    flat = np.concatenate([g.ravel() for g in gs])
    assert math.isclose(norm, float(np.linalg.norm(flat)), rel_tol=1e-14)
    clipped = np.concatenate([(g * scale).ravel() for g in gs])
    assert math.isclose(float(np.linalg.norm(clipped)), 0.5 * norm / (norm + 1e-6),
                        rel_tol=1e-14)
    assert np.linalg.norm(clipped) <= 0.5


def test_clip_scale_special_values():
    assert clip_scale([np.zeros(4)], 1.0) == (1.0, 0.0)
    s, n = clip_scale([np.array([1.0, np.nan])], 1.0)
    assert math.isnan(s) and math.isnan(n)
    s, n = clip_scale([np.array([1.0, np.inf])], 1.0)
    assert s == 0.0 and n == math.inf


def _with_clip(cfg, max_norm):
    cfg = dict(cfg)
    cfg["opt"] = dict(cfg["opt"], clip_norm=max_norm)
    return cfg


def test_first_sgd_step_closed_form():
    """theta_1 = theta_0 - lr * (s g + wd theta_0) with s from the unclipped
    gradient g of step 1 (momentum buffer starts at 0)."""
    cfg = get_config("mlp3")
    plain = run(cfg, "eager", steps=1, snapshots=(0, 1))
    g = plain["snapshots"][1]["grad"]
    norm = float(np.linalg.norm(np.concatenate([g[k].ravel() for k in g])))
    max_norm = 0.25 * norm
    s = max_norm / (norm + 1e-6)
    clipped = run(_with_clip(cfg, max_norm), "eager", steps=1, snapshots=(0, 1))
    assert math.isclose(clipped["clips"][0][0], s, rel_tol=1e-14)
    lr, wd = cfg["opt"]["lr"], cfg["opt"]["weight_decay"]
    for k, th0 in clipped["snapshots"][0]["params"].items():
        want = th0 - lr * (s * g[k] + wd * th0)
        np.testing.assert_allclose(clipped["params"][k], want, rtol=1e-13, atol=1e-15,
                                   err_msg=k)


def _same(a, b):
    for key in ("params", "m", "v"):
        for n in a[key]:
            np.testing.assert_array_equal(a[key][n], b[key][n], err_msg=f"{key}[{n}]")
    np.testing.assert_array_equal(a["losses"], b["losses"])
    assert a["eval_loss"] == b["eval_loss"]
    assert a["step"] == b["step"]


@pytest.mark.parametrize("name", ["mlp3", "mlp8x1024", "tblock12"])
def test_clipped_orderings_bit_identical(name):
    cfg = reduced_config(name)
    plain = run(cfg, "eager", steps=1, snapshots=(1,))
    g = plain["snapshots"][1]["grad"]
    norm = float(np.linalg.norm(np.concatenate([g[k].ravel() for k in g])))
    c = _with_clip(cfg, 0.5 * norm)      # clips at least the first step
    e = run(c, "eager")
    f = run(c, "ff")
    _same(e, f)
    assert e["clips"] == f["clips"]
    assert e["clips"][0][0] < 1.0
    # clipping changed the trajectory
    u = run(cfg, "eager")
    assert any(np.any(e["params"][k] != u["params"][k]) for k in u["params"])
    with pytest.raises(ValueError):
        run(c, "bf")


def test_inactive_clip_is_identity():
    cfg = reduced_config("mlp8x1024")
    u = run(cfg, "eager")
    c = run(_with_clip(cfg, 1e30), "ff")
    _same(u, c)
    assert all(s == 1.0 for s, _ in c["clips"])
