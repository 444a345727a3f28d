"""Seeded synthetic inputs shared by the oracle tests, the GPU parity tests and
the benchmark.

This module holds no arithmetic of the method itself: it only names the
workload shapes and draws seeded random tensors.  Every tensor is drawn in
float32 from numpy's PCG64 generator (seeded with ``[seed, stream_id]`` so each
tensor has its own stream), scaled by its standard deviation and rounded to
bfloat16 with round-to-nearest-even when the workload is bf16.  Both the CPU
oracle and the GPU path consume exactly these bits.
"""
from .gen import (Workload, WORKLOADS, random_block_mask, bf16_bits_from_f32, f32_from_bf16_bits,
                  draw, draw_int)

__all__ = ["Workload", "WORKLOADS", "random_block_mask", "bf16_bits_from_f32", "f32_from_bf16_bits",
           "draw", "draw_int"]
