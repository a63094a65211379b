"""CPU oracle of the routed-expert FP8 MoE FFN (test infrastructure only).

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s
``cpu_baseline`` leg may import this package; the GPU library never does.
"""
from .moe_oracle import (  # noqa: F401
    BLOCK, E4M3_MAX, E4M3_TABLE, e4m3_decode, e4m3_encode, bf16_to_f32, f32_to_bf16,
    quantize_rows, quant_act, quantize_weight, quantize_experts, check_routing, permute,
    block_scaled_matmul, silu_mul, expert_rows, expert_ffn, combine, prepare_weights,
    moe_layer, moe_layer_dense, block_scaled_matmul_w8a16, expert_rows_w8a16, expert_ffn_w8a16,
    moe_layer_w8a16,
)
