"""Seeded synthetic inputs for the block-memory attention path.

This package only draws numbers. It holds none of the attention method's
arithmetic; both the device library's tests/benchmark and the CPU oracle take
their inputs from here.
"""
from .synth import WORKLOADS, Workload, Synth, bf16_bits_to_f32, f32_to_bf16_bits

__all__ = ["WORKLOADS", "Workload", "Synth", "bf16_bits_to_f32", "f32_to_bf16_bits"]
