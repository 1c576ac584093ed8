"""CPU oracle for the pruned layer stack -- test infrastructure only.

Imported by the tests, the smoke check and the benchmark's CPU-baseline leg;
never by the library or its binding.
"""
from .zsa_oracle import (  # noqa: F401
    DECODER, ENCODER, LayerCfg, attention, bf16_round, gelu, keep_count, keep_schedule,
    layer_forward, layer_norm, rms_norm, rope, select_topk, sequence_layer, silu,
    stack_forward,
)
