"""Seeded synthetic workloads shared by the oracle tests, the GPU tests and the benchmark."""
from .workloads import (CONFIGS, Layer, LayerConfig, bf16_bits_to_f32, f32_to_bf16_bits,
                        full_width_weights, make, round_to_bf16, routing_targets)

__all__ = ["CONFIGS", "Layer", "LayerConfig", "bf16_bits_to_f32", "f32_to_bf16_bits",
           "full_width_weights", "make", "round_to_bf16", "routing_targets"]
