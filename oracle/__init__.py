"""CPU oracle for the mask-aware K/V-cached block stack (test infrastructure only).

Only the tests, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package. It shares no code with the GPU path.
"""
from .stack import (  # noqa: F401
    attention_head,
    bf16_round,
    block_rows,
    compact,
    dense_stack,
    gelu,
    layer_flops,
    layer_norm,
    linear,
    masked_rows_of_stack,
    masked_stack,
    masked_tokens,
    rounder,
)
from .planner import best_dense_prefix, greedy_choice, pipeline_latency  # noqa: F401
from .routing import CostModel, batch_latency, block_costs, calc_cost, fit_linear, route  # noqa: F401
from .ycache import dense_inputs, kv_cache_of_inputs, kv_of_inputs, masked_stack_y  # noqa: F401
