"""Seeded synthetic workloads shared by the tests, the bench and the oracle checks.

Holds shapes and random streams only; neither the GPU path nor the oracle is
imported from here.
"""
from .configs import DrafterConfig, NAMED, prefix_range  # noqa: F401
from . import configs  # noqa: F401
from .gen import (Inputs, LayerWeights, UpdateRows, Weights, float_tensor, make_inputs,  # noqa: F401
                  make_uniforms, make_update_rows,
                  make_prefix_lens, make_weights, to_f64)
