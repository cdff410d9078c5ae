"""Seeded synthetic inputs shared by the tests, the bench and the smoke check.

This module holds no arithmetic of the attention method: it only draws
random tensors and describes workload shapes (segment lists, head counts,
value scales).  Both the oracle side and the GPU side consume what it
returns; neither side is imported here.

Inputs are drawn in float32 from a CPU ``torch.Generator`` and rounded to
bfloat16 (round to nearest even), so every consumer sees the same bf16 bits.
"""
from .workloads import (  # noqa: F401
    ANCHOR, TEXT, TARGET, REF, KIND_NAMES, Workload, WORKLOADS, workload,
    derive_seed, bf16_normal, draw_qkv, SCALING_KS, draw_chain_weights, draw_hidden,
)
