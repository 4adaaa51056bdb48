"""Seeded synthetic GQA decode inputs shared by the oracle tests, the GPU tests and the bench.

This package draws random keys, values and queries and rounds them to bf16. It holds none of
CompKV's arithmetic (no block statistics, scores, selection or attention), so that the CPU oracle
and the HIP path can both consume its output without sharing any code of the method.
"""
from .gqa_decode import (  # noqa: F401
    Workload,
    WORKLOADS,
    bf16_bits_to_f32,
    f32_to_bf16_bits,
    gen_unit_kv,
    gen_queries,
    gen_layer,
    offset_blocks,
)
