"""Seeded synthetic inputs for LM-GC workloads.

This package holds only workload descriptions (model shapes, serialisation
parameters, value distributions) and seeded generators of the inputs: gradient
vectors and random-init decoder weights.  It contains none of the method's
arithmetic (no serialisation, no lossy sparsification or quantisation, no
forward pass, no coding) and it is the only code that both the CPU oracle
and the GPU library's tests/bench use.
"""
from .configs import (ModelShape, SerialSpec, Workload, WORKLOADS, get_workload,
                      hex_serial, parse_lossy, lossy_bytes_per_value, LOSSY_VARIANTS)
from .gen import (gen_values, gen_weights, weight_manifest, bf16_bits_to_f32,
                  f32_to_bf16_bits)

__all__ = ["ModelShape", "SerialSpec", "Workload", "WORKLOADS", "get_workload",
           "hex_serial", "parse_lossy", "lossy_bytes_per_value", "LOSSY_VARIANTS",
           "gen_values", "gen_weights", "weight_manifest",
           "bf16_bits_to_f32", "f32_to_bf16_bits"]
