"""Seeded synthetic inputs shared by the CPU oracle and the GPU path.

This package holds the workload shapes and the random-number recipe only; it
contains none of the DiT block's or the denoising step's arithmetic.  Both sides of every parity check
read the exact same stored bits from here.
"""
from .workloads import (
    Workload, WORKLOADS, get_workload, ModelWorkload, MODEL_WORKLOADS, get_model_workload,
    RequestClass, REQUEST_CLASSES, MODEL_SHAPES, SP_DEGREES, share_workload,
)
from .trace import make_trace, cost_matrix, read_cost_table, standalone_us
from .gen import (
    bf16_bits, generate_block_inputs, generate_tensor, TensorSpec, draw,
    block_tensor_specs, generate_attention_inputs, generate_sampled_rows,
    model_tensor_specs, generate_model_inputs, MODEL_WEIGHT_NAMES,
)

__all__ = [
    "Workload", "WORKLOADS", "get_workload", "bf16_bits", "generate_block_inputs",
    "generate_tensor", "TensorSpec", "block_tensor_specs",
    "generate_attention_inputs", "generate_sampled_rows", "draw",
    "ModelWorkload", "MODEL_WORKLOADS", "get_model_workload", "model_tensor_specs",
    "generate_model_inputs", "MODEL_WEIGHT_NAMES", "RequestClass", "REQUEST_CLASSES", "MODEL_SHAPES",
    "SP_DEGREES", "share_workload", "make_trace", "cost_matrix", "read_cost_table", "standalone_us",
]
