"""Seeded synthetic inputs shared by the fp64 oracle and the HIP path.

This package draws random numbers and builds masks; it performs none of the
method's arithmetic (no dilation, ranking, attention or bank placement).  Both
sides of every parity check consume the exact arrays produced here.
"""
from .gen import (  # noqa: F401
    CONFIGS, Config, Weights, FrameInputs, Sequence,
    bf16_bits, bits_to_f32, to_storage, storage_to_f64,
    ellipse_mask, make_weights, make_frame, make_sequence, make_rope_table, make_decoder_logits, k_from_rho,
    fall_counts, make_stack_weights, STACK_MATRICES, STACK_NORMS,
)
