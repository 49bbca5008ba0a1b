"""Seeded synthetic inputs shared by the oracle and the HIP path.

This package draws random numbers and encodes them as bf16 bit patterns
(uint16) or fp32 arrays. It holds none of the method's arithmetic: no
gather, no product, no reduction, no schedule and no model.
"""
from .gen import (  # noqa: F401
    CONFIGS,
    bf16_bits,
    config_shapes,
    make_ag_inputs,
    make_rs_inputs,
    make_int_ag_inputs,
    make_int_rs_inputs,
    make_config_inputs,
    make_int_config_inputs,
)
