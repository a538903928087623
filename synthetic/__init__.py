"""Seeded synthetic inputs shared by the CPU oracle and the GPU path.

This module draws random numbers and holds the model shapes; it contains none
of the forward pass's arithmetic.  Both sides receive the tensors it returns as
plain inputs, so nothing here is computed by either implementation.
"""
from .models import (MODEL_SHAPES, WORKLOADS, small_shape, model_weights,
                     weight_names, weight_shapes, prompts, paged_workload, is_moe_layer)

__all__ = ["MODEL_SHAPES", "WORKLOADS", "small_shape", "model_weights",
           "weight_names", "weight_shapes", "prompts", "paged_workload", "is_moe_layer"]
