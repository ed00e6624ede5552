"""Seeded synthetic inputs for the routed-expert MoE hot path.

This package only draws random numbers and stores them in the formats the
kernels consume (bf16 bit patterns, OCP fp8-e4m3 codes with fp32 block
scales).  It holds none of the method's arithmetic: no gating, no
permutation, no expert FFN and no combine.  Both the CPU oracle and the GPU
path read their inputs from here.
"""
from .gen import (  # noqa: F401
    CONFIGS,
    MoEConfig,
    LayerInputs,
    PhaseInputs,
    make_layer,
    make_phase,
    make_weights,
    custom_config,
    bf16_bits,
    e4m3_codes,
    E4M3_MAX,
)
