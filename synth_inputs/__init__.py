"""Seeded synthetic inputs for the CAEE MoE-layer workloads.

This package is shared by the fp64 oracle and by the HIP path: it only draws
random numbers and encodes them into storage formats (fp32, bf16 bits, OCP
e4m3 codes with block scales). None of the method's arithmetic (routing,
pruning, compensation, expert FFN) lives here.
"""
from .layers import (  # noqa: F401
    LayerShape,
    TINY_F32,
    R1_BF16,
    R1_FP8,
    WORKLOADS,
    RoutingInputs,
    make_routing_inputs,
    make_call_sequence,
    popularity_ranks,
    make_cost_table,
    make_bins,
    make_expert_weights_np,
    make_expert_weights_torch,
    bf16_bits_from_f32,
    weight_bytes_per_expert,
)
