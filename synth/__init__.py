"""Seeded synthetic workloads for the modality-aware W8A8 + low-rank linear.

This package only draws random inputs (activations, modality layouts, float
weights).  It contains none of the quantization or compensation arithmetic, so
both the CPU oracle and the GPU path can consume its outputs without sharing
any of the method's code.
"""
from .workloads import (  # noqa: F401
    CONFIGS,
    LayerInputs,
    Projection,
    make_layer_inputs,
    make_modality_layout,
    make_weight,
    make_activations,
    config_by_name,
)
