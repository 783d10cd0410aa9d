"""fp64 CPU oracle of the fused MoE layer -- test infrastructure only.

Only the tests, the smoke check and the CPU-baseline leg of the benchmark may
import this package; the HIP library and its binding never do.
"""
from .moe_oracle import (  # noqa: F401
    bf16_to_f64, f32_to_bf16_rne, e4m3_decode, e4m3_encode, int4_unpack,
    dequant_weight, gate, permute, permute_capacity, act_quant_fp8,
    act_dequant_fp8, act_quant_mxfp8, act_dequant_mxfp8, swiglu_expert, activation_operand, forward,
)
