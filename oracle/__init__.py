"""CPU oracle for the ExactMoE routed-expert layer (test infrastructure only).

Only the test-suite, the package smoke check and the benchmark's CPU-baseline
leg may import this package.  The product path never does.
"""
from .exactmoe_oracle import *  # noqa: F401,F403
from .exactmoe_oracle import (GROUP, QuantizedExpert, Routing, Grouping, SlotCache,
                              ScaleRangeError, quantize_matrix, dequantize_matrix,
                              quantize_expert, packed_pool_bytes, router_logits,
                              topk_experts, mixture_weights, group_by_expert,
                              plan_waves, silu, expert_mlp, route, moe_forward,
                              pair_outputs)
