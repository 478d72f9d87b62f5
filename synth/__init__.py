"""Seeded synthetic inputs shared by the oracle and the GPU path's tests and bench.

This package draws random tensors and prepares them the way the workloads
describe them (normal draws, per-row RMS normalisation of queries and keys,
round-to-nearest-even to bfloat16). It holds none of the attention arithmetic.
"""
from .inputs import (  # noqa: F401
    Workload,
    WORKLOADS,
    bf16_bits_to_f32,
    f32_to_bf16_bits,
    draw_tensor,
    draw_qkv_sequence,
    draw_chunk,
    AudioWorkload,
    AUDIO_WORKLOADS,
    face_ids,
    draw_audio,
)
