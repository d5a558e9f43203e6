"""Seeded synthetic inputs for the workloads (shared by the oracle and the GPU path).

Every array is drawn in float64 by numpy's PCG64 generator and rounded to
float32, so both sides start from bit-identical values.  Each draw has its own
generator seeded by SeedSequence([seed, purpose, index]), so any batch can be
made on its own without drawing the ones before it:

  purpose 0  parameter number `index` in model order
  purpose 1  training batch number `index` (1-based step)
  purpose 2  the evaluation batch

Value distributions (per workload description): inputs and regression targets
N(0, 1); labels uniform integers in [0, classes); weights uniform on
+-sqrt(6 / fan_in) (Kaiming-uniform); biases and LayerNorm shifts 0;
LayerNorm scales 1.
"""
import numpy as np

from .configs import param_specs, input_shape, output_shape

_PARAMS, _BATCH, _EVAL = 0, 1, 2


def _rng(seed, purpose, index):
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, purpose, index])))


def make_params(cfg, seed=0):
    """Initial parameters: dict name -> float32 array, in model order."""
    out = {}
    for idx, (name, shape, init, fan_in) in enumerate(param_specs(cfg)):
        if init == "kaiming":
            bound = np.sqrt(6.0 / fan_in)
            out[name] = _rng(seed, _PARAMS, idx).uniform(-bound, bound, size=shape).astype(np.float32)
        elif init == "zeros":
            out[name] = np.zeros(shape, np.float32)
        elif init == "ones":
            out[name] = np.ones(shape, np.float32)
        else:
            raise ValueError(init)
    return out


def _batch(cfg, rng):
    x = rng.standard_normal(size=input_shape(cfg)).astype(np.float32)
    if cfg["loss"] == "xent":
        y = rng.integers(0, cfg["classes"], size=(cfg["batch"],), dtype=np.int64)
    else:
        y = rng.standard_normal(size=output_shape(cfg)).astype(np.float32)
    return x, y


def make_batch(cfg, step, seed=0):
    """Training batch for 1-based `step`: (inputs float32, labels int64 | targets float32)."""
    return _batch(cfg, _rng(seed, _BATCH, step))


def make_eval_batch(cfg, seed=0):
    """The fixed evaluation batch."""
    return _batch(cfg, _rng(seed, _EVAL, 0))
