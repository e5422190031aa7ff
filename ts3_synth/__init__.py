"""Seeded synthetic inputs (points, features, weights) shared by the oracle's
tests and the GPU path's tests and benchmark.  Holds none of the layer's own
arithmetic."""
from .features import bf16_bits_to_f32, f32_to_bf16_bits, round_bf16, to_f32
from .weights import make_block_weights, make_weights
from .workloads import WORKLOADS, Workload, features, round_storage

__all__ = ["WORKLOADS", "Workload", "features", "make_block_weights", "make_weights", "round_bf16", "round_storage",
           "to_f32", "f32_to_bf16_bits", "bf16_bits_to_f32"]
