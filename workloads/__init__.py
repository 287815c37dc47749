"""Seeded synthetic workloads for the branch-parallel decode step.

This package only draws inputs: page/branch structure and the Q/K/V (and, for
the decoder-stack workload, weight and hidden-state) values.  It holds none of
the method's arithmetic, so both the fp64 oracle and the GPU path consume the
exact same stored bits without sharing any computation.
"""
from .configs import CONFIGS, get_config  # noqa: F401
from .gen import (  # noqa: F401
    AttnBatch,
    DecodeInputs,
    bf16_bits_to_f64,
    f64_to_bf16_bits,
    make_attn_batch,
    make_decode_inputs,
    make_pmtp_inputs,
    make_structure,
)
