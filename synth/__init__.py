"""Seeded synthetic layers and the round-to-nearest host quantizer.

This package produces the inputs of one refinement problem: the original
weights W, the calibration Hessian H = X^T X / n + damping * I, and a host
state (codes, scales, zero points).  It holds none of the refinement
arithmetic; both the HIP path and the float64 oracle consume what it makes.
"""

from .layers import (CONFIGS, LayerConfig, calibration_chunks, make_hessian, make_layer,
                     make_weights, propagated_inputs)
from .rtn import rtn_quantize

__all__ = ["CONFIGS", "LayerConfig", "calibration_chunks", "make_layer", "make_weights",
           "make_hessian", "propagated_inputs", "rtn_quantize"]
