"""CPU oracle for the MoE expert stage.

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, ``__graft_entry__.smoke()``
and the CPU-baseline leg of ``bench.py``, never by the product package.
It is a plain fp64 statement of what the stage computes and shares no code
with the HIP path.
"""
from .moe_oracle import (  # noqa: F401
    dispatch, bf16_bits_to_f64, bf16_bits_to_f32, round_f32_to_bf16, e4m3_decode, e4m3_encode,
    quantize_groups, dequantize_groups, dequantize_blocks, silu, swiglu_ffn,
    OracleWeights, stage_inputs_x, run_stage, rel_l2, E4M3_TABLE, E4M3_MAX,
    grouped_counts, run_grouped,
)
