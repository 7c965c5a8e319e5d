"""Seeded synthetic inputs for the CateKV hybrid-KV decode path.

This package only draws random numbers and lays them out: it holds none of
the method's arithmetic (no softmax, no scoring, no selection).  Both the CPU
oracle and the GPU path are fed from it, so it imports neither.
"""
from .gen import (  # noqa: F401
    WORKLOADS,
    Workload,
    SequenceInputs,
    bf16_bits_to_f32,
    f32_to_bf16_bits,
    decode_queries,
    make_sequence,
    sequence_lengths,
    storage_to_f64,
)
