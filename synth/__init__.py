"""Seeded synthetic workloads (shapes, distributions, streams) for the
refine + verify path.  Holds no arithmetic of the method; the oracle and the
device path both take their inputs from here."""
from .configs import WORKLOADS, BY_NAME, Workload, scaled  # noqa: F401
from .gen import (make_weights, make_inputs, Inputs, as_f32,  # noqa: F401
                  f32_to_bf16_bits, bf16_bits_to_f32, make_layer_weights,
                  make_layer_inputs, LayerInputs, LAYER_SHAPES)
