"""Seeded synthetic inputs for one GPU's share of an expert-parallel MoE layer.

This package only draws and shapes inputs; it holds none of the layer's
arithmetic. Both the CPU oracle (``oracle/``) and the HIP path consume what it
produces, so it must stay independent of both.
"""
from .moe_inputs import (  # noqa: F401
    CONFIGS,
    LayerInputs,
    LayerShape,
    make_activation_matrix,
    make_layer,
    make_router,
    make_experts,
    router_grid_q,
    round_to_bf16_values,
)
