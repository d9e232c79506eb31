"""Seeded synthetic workloads for the per-micro-step MoE expert layer.

This package produces inputs only: routing ids and gates shaped like RL
micro-step routing, token activations, expert weights, upstream gradients,
and a per-micro-step placement plan standing in for the paper's planner
(Sec. 7, Alg. 1 and Alg. 3). It holds none of the expert layer's own
arithmetic; both the CPU oracle and the HIP path consume what it returns.
"""
from .bf16 import bf16_round, f32_to_bf16_bits, bf16_bits_to_f32
from .synth import (
    ConfigSpec,
    CONFIGS,
    CONFIG_IDS,
    Plan,
    MicroStep,
    Workload,
    make_workload,
    make_custom,
    plan_from_slots,
)

__all__ = [
    "bf16_round",
    "f32_to_bf16_bits",
    "bf16_bits_to_f32",
    "ConfigSpec",
    "CONFIGS",
    "CONFIG_IDS",
    "Plan",
    "MicroStep",
    "Workload",
    "make_workload",
    "make_custom",
    "plan_from_slots",
]
