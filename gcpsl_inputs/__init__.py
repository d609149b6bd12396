"""Seeded synthetic inputs shared by the oracle and the HIP path.

This package holds workload descriptions and seeded input generators only:
the image set, its labels, the Dirichlet split of examples over clients and
the initial parameter vector.  It contains none of the method's arithmetic
(no assignment rule, no sampler, no layer, no update, no fusion), so both
the CPU oracle and the GPU path can take their inputs from it without
sharing any computation.
"""
from .configs import CONFIGS, get_config, model_layers, norm_layout, param_layout, param_counts
from .synth import make_dataset, init_norm_state, init_params, client_stats

__all__ = [
    "CONFIGS", "get_config", "model_layers", "norm_layout", "param_layout", "param_counts",
    "make_dataset", "init_norm_state", "init_params", "client_stats",
]
