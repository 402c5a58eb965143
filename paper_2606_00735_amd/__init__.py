"""One GPU's share of an expert-parallel MoE layer on MI355X (gfx950).

The computation ViBE (arXiv 2606.00735) balances across GPUs: top-k gating,
the per-expert activation profile, dispatch permutation, grouped SwiGLU
expert FFN, weighted combine, and the per-expert latency-vs-load sweep from
which the per-GPU performance model f_g(n) is fitted, and ViBE's placement
control path on top of it (latency-aware greedy placement, drift detector,
incremental swap solver), and an MXFP8 (FP8 E4M3 with E8M0 block
scales) variant of the expert FFN. Every step runs in the
HIP kernels of ``libmoe.so`` (C ABI in ``include/moe.h``); this package only
marshals torch tensors into those calls.
"""
from ._lib import (  # noqa: F401
    EXPORTED,
    FFN_COUNTER_BYTES,
    LIB_PATH,
    MoeError,
    MxTensor,
    ffn_hidden,
    ffn_mx_ws_bytes,
    ffn_ws_bytes,
    gate_ws_bytes,
    hist_ws_bytes,
    load_library,
    moe_drift_distance,
    moe_expert_histogram_scan,
    moe_fit_latency_model,
    moe_gate_topk,
    moe_grouped_gemm_mx,
    moe_grouped_swiglu_ffn,
    moe_grouped_swiglu_ffn_gather,
    moe_grouped_swiglu_ffn_mx,
    moe_grouped_swiglu_ffn_noalloc,
    moe_grouped_swiglu_mx,
    moe_layer,
    moe_load_sweep,
    moe_load_sweep_mx,
    moe_mx_quantize,
    moe_permute,
    moe_place_greedy,
    moe_place_incremental,
    moe_placement_cost,
    moe_unpermute_combine,
    moe_window_push,
    pad_weight_rows,
    weight_row_stride,
)
