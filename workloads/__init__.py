"""Seeded synthetic workloads for the integrated fixed-point quantized conv path.

This package is shared by the oracle, the tests and the benchmark. It only
describes layer stacks (explicit shapes) and draws seeded random tensors; it
holds none of the method's arithmetic (no convolution, normalisation,
threshold folding or pooling).
"""
from .stacks import CONFIGS, Conv, Pool, get_stack, stack_names
from .gen import (SEED_ROOT, Kind, layer_params, stack_input, quant_thresholds,
                  input_step)

__all__ = ["CONFIGS", "Conv", "Pool", "get_stack", "stack_names", "SEED_ROOT",
           "Kind", "layer_params", "stack_input", "quant_thresholds",
           "input_step"]
