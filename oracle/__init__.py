"""CPU oracle for the routed-expert MoE hot path -- TEST INFRASTRUCTURE ONLY.

Only the test-suite, the smoke check and the benchmark's CPU-baseline leg may
import this package.  The product path (the HIP library and its Python
binding) never imports, calls or links anything here, and this package shares
no code with it.  See moe.py for what each function computes and which part
of the paper it follows.
"""
from .moe import (  # noqa: F401
    bf16_to_f64,
    e4m3_to_f64,
    e4m3_quantize,
    quantize_rows,
    dequant_rows,
    dequant_weight,
    route,
    permute,
    permute_masked,
    expert_ffn,
    expert_hidden,
    expert_down,
    grouped_hidden,
    grouped_down,
    grouped_ffn,
    combine,
    moe_local_share,
    token_output,
    x_moe,
    decode_quota,
    count_tiles,
    PermuteResult,
)
