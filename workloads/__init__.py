"""Seeded synthetic inputs for the speculative-decoding verify step.

This package only draws random numbers and lays them out in the memory
formats the verify step consumes (bf16 bit patterns, fp32 logits, int32
lengths). It holds none of the verify step's arithmetic: no softmax, no
acceptance rule, no attention. Both the CPU reference and the HIP path are
fed from here.
"""

from .configs import CONFIGS, ChainShape, VerifyShape, get_config, small_shape
from .gen import (
    LevelInputs,
    bf16_bits_from_f32,
    chain_inputs,
    kv_slab,
    level_inputs,
    logits_rows,
    q_block,
)

__all__ = [
    "CONFIGS",
    "ChainShape",
    "VerifyShape",
    "get_config",
    "small_shape",
    "LevelInputs",
    "bf16_bits_from_f32",
    "chain_inputs",
    "kv_slab",
    "level_inputs",
    "logits_rows",
    "q_block",
]
