"""Fused Mixture-of-Experts layer for AMD MI355X (gfx950).

MoE Gate -> Fused MoE -> Weight Sum (the paper's MoE skeleton, Fig. 1 and
Fig. 3) as hand-written HIP kernels behind the C ABI of include/moe.h (plus
the achievable-peak probes of include/moe_peaks.h); this package is the thin
Python binding over that library (``_binding``) and its build script
(``build``).
"""
from ._binding import (  # noqa: F401
    LIB_PATH, NUM_STAGES, STAGES, MoeArgs, MoeError, lib, make_args, moe_act_quant_fp8, moe_forward,
    STATIC_WS_BYTES, moe_forward_args, moe_forward_profiled, moe_forward_static_ws, moe_gate_topk, moe_permute, moe_permute_capacity,
    moe_router_gate_topk,
    moe_permute_workspace_bytes, moe_workspace_bytes, moe_workspace_layout,
    moe_peak_copy, moe_peak_mfma, moe_peak_mfma_flops_per_launch, moe_peak_read, moe_peak_sink_elems,
    moe_peak_lds_copy, moe_peak_lds_copy_bytes_per_launch, moe_peak_lds_read, moe_peak_lds_read_bytes_per_launch,
)
