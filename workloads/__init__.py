"""Seeded synthetic workloads for the budget-adapted prefill.

This package only *describes* and *draws* inputs: model shapes, batch shapes,
vision-token scores, hidden states, weights and the layer / head / FFN masks.
It holds none of the method's arithmetic, so both the GPU path's tests and the
CPU oracle can take their inputs from it without sharing any computation.
"""
from .configs import ModelShape, Workload, WORKLOADS, HEADLINE, get_workload, keep_count, scaled
from .generate import (
    CONTROLLER_NAMES, WEIGHT_NAMES, ControllerDraw, Inputs, as_f32, draw_controller, draw_hidden,
    draw_inputs, draw_layer_weights, draw_masks, draw_scores, round_to_bf16, storage_dtype,
)

__all__ = [
    "ModelShape", "Workload", "WORKLOADS", "HEADLINE", "get_workload", "keep_count", "scaled",
    "CONTROLLER_NAMES", "ControllerDraw", "draw_controller", "WEIGHT_NAMES", "Inputs", "as_f32",
    "draw_hidden", "draw_inputs", "draw_layer_weights", "draw_masks", "draw_scores",
    "round_to_bf16", "storage_dtype",
]
