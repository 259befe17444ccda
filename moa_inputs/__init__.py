"""Seeded synthetic inputs shared by the HIP engine's harness and the oracle.

This package only draws random numbers and lays them out: model weights,
query prompts, expert routing, per-request generation budgets. It contains
none of the method's arithmetic (no transformer maths, no scheduling), so the
oracle and the product path can both consume it without sharing code.
"""
from .configs import CONFIGS, ModelShape, EngineConsts, config
from .weights import (TENSOR_NAMES, tensor_shapes, generate_weights,
                      pack_blob, bf16_bits_to_f32, f32_to_bf16_bits)
from .workload import Workload, make_workload, StragglerWorkload, make_straggler_workload

__all__ = ["CONFIGS", "ModelShape", "EngineConsts", "config", "TENSOR_NAMES",
           "tensor_shapes", "generate_weights", "pack_blob", "bf16_bits_to_f32",
           "f32_to_bf16_bits", "Workload", "make_workload",
           "StragglerWorkload", "make_straggler_workload"]
