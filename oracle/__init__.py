"""CPU oracle of the Chimera decode step -- test infrastructure only.

Only tests, the smoke entry point and the benchmark's CPU-baseline leg may
import this package.  The GPU product path never imports or calls it.
"""
from .chimera_oracle import (  # noqa: F401
    Decoder, Forcing, Oracle, Tree, apply_rope, argmax_lowest, bf16_bits_to_f32,
    masked_attention, rms_norm, rope_cos_sin, round_bf16, silu, softmax_rows, top_s)
