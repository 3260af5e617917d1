"""fp64 CPU oracle for the stage-shard forward/backward.

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the
benchmark's CPU-baseline leg, never by the HIP library or its binding.
"""
from .stage import (  # noqa: F401
    GELU_A, GELU_C, block_backward, block_forward, causal_attention_backward,
    causal_attention_forward, gelu, gelu_grad, layer_norm_backward, layer_norm_forward,
    shard_block, shard_run, stage_backward, stage_forward, zero_pad_block,
)
