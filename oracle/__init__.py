"""CPU oracle of the SonicMoE layer (arXiv 2512.14080) -- TEST INFRASTRUCTURE ONLY.

A plain, slow, obviously-correct NumPy implementation of what the MoE layer
computes: router scores, token-choice top-K routing, routing metadata, token
rounding (Section 5.2 and the appendix on rounding subroutines), the forward
pass (Section 3, forward algorithm) and the backward pass (Section 3 and the
"Gradient computation" appendix), plus the router backward.

Only the test-suite, the smoke check and the benchmark's CPU-baseline leg may
import this package.  The HIP product path never calls, links or imports it,
and it shares no code with the HIP path: the only common dependency is the
seeded input generator, which holds none of the method's arithmetic.

Arithmetic runs in fp32 by default (the precision fixed for the oracle of this
layer) and in fp64 when ``dtype=np.float64`` is passed (used by the pins).
"""
from .routing import (router_logits, softmax_scores, topk_select, tc_membership,
                      routing_from_membership, round_tokens, route)
from .layer import (swiglu, dswiglu, forward, backward, forward_tokens, backward_tokens,
                    weight_grad_columns, cached_bytes)

__all__ = [
    "router_logits", "softmax_scores", "topk_select", "tc_membership",
    "routing_from_membership", "round_tokens", "route",
    "swiglu", "dswiglu", "forward", "backward", "forward_tokens", "backward_tokens",
    "weight_grad_columns", "cached_bytes",
]
