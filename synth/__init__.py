"""Seeded synthetic inputs for the fused MoE layer (data only, no layer arithmetic)."""
from .moe_inputs import (  # noqa: F401
    MoeConfig,
    CONFIGS,
    config,
    tiny_config,
    make_inputs,
    make_routing_inputs,
    to_device,
    make_expert_weights,
    make_router_weights,
)
