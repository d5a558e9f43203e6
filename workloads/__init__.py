"""Synthetic workloads shared by the oracle and the HIP path.

This package describes the five training workloads as data (layer shapes,
optimizer hyperparameters, batch sizes) and draws every seeded input from
them: initial parameters, input batches, labels and targets.  It holds none
of the method's arithmetic (no layer, loss or optimizer math); the oracle and
the GPU path each implement that on their own.
"""
from .configs import (CONFIGS, get_config, reduced_config, param_specs, describe,  # noqa: F401
                      mlp_ties, mbv2_blocks)
from .gen import make_params, make_batch, make_eval_batch  # noqa: F401
