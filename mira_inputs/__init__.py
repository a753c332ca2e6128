"""Seeded synthetic inputs for the Mira MoE expert step.

This module only draws random tensors of the workloads' shapes and
distributions; it holds none of the method's arithmetic.  Both the GPU
library's tests/benchmark and the CPU oracle are fed from it, so the two
sides always see the same bytes.

Every tensor comes from its own torch generator whose seed is derived from
(workload, layer, expert, tensor) through numpy's SeedSequence, so any single
expert of any layer can be regenerated alone, on the host or on the device.
"""
from .configs import CONFIGS, MoEConfig, get_config  # noqa: F401
from .gen import (  # noqa: F401
    activations,
    drift_bias,
    drift_hot,
    router_weights,
    router_bias,
    expert_weights,
    predictor_weights,
    mixture_weights,
    routing_sample,
    resident_experts,
    tensor_seed,
)
