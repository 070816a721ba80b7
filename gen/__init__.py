"""Seeded synthetic inputs shared by the oracle, the tests and the benchmark.

This package holds no part of the compression method: it only draws weights
and activation vectors with the shapes and value distributions of decoder-layer
projections, and rounds them to bfloat16 (or float16) bit patterns.
"""
from .synth import (WORKLOADS, MatrixSpec, workload_matrices, gen_matrix, gen_matrix_device, gen_x,
                    f32_to_bf16_bits, bf16_bits_to_f32, bf16_bits_to_f16_bits, random_bf16,
                    random_fp16, random_x)

__all__ = ["WORKLOADS", "MatrixSpec", "workload_matrices", "gen_matrix", "gen_matrix_device", "gen_x",
           "f32_to_bf16_bits", "bf16_bits_to_f32", "bf16_bits_to_f16_bits", "random_bf16",
           "random_fp16", "random_x"]
