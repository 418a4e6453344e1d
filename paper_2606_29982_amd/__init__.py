"""MI355X-native CAEE (Cost-Aware Expert Execution) MoE-layer hot path.

The layer runs in hand-written gfx950 HIP kernels behind the C ABI declared
in include/caee.h (libcaee.so); ``caee`` is its Python binding.
"""
from .caee import (  # noqa: F401
    CaeeError, Layer, abi_version, alloc_route_out, alloc_workspace, expert_ffn, moe_layer,
    route_prune, timing_enable, timing_query, timing_reset, workspace_size, Offload, lru_step)
