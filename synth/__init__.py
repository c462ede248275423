"""Seeded synthetic workloads for the Domino drafting path.

This module only draws inputs: configuration presets, random weights, context
KV caches, anchor tokens and target logits.  It performs none of the method's
arithmetic, so both the CPU oracle and the GPU path can be fed from it without
sharing any computation.
"""
from .configs import DominoConfig, PRESETS, get_config  # noqa: F401
from .inputs import (  # noqa: F401
    bf16_round,
    make_weights,
    make_inputs,
    make_target_logits,
    make_random_topk,
    make_forced_tokens,
    make_append_hidden,
    make_target_weights,
    weight_shapes,
    head_param_count,
)
