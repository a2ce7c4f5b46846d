"""Seeded synthetic inputs shared by the oracle-side tests and the GPU path.

This package only draws and encodes input tensors (random numbers, masks,
bf16 rounding of the drawn values). It holds none of the method's
arithmetic: no activity test, no statistic, no score, no selection.
"""
from .gen import (  # noqa: F401
    TEXT, IMAGE, VIDEO, AUDIO, MODALITY_NAMES,
    Segment, Workload, default_params, make_workload, f32_to_bf16_bits,
    bf16_bits_to_f32, CONFIG_NAMES, DRAFT_ROWS, DRAFT_VOCAB, draft_logits, simhash_planes,
)
