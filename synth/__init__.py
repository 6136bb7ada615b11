"""Seeded synthetic inputs for the LoGo attention layer.

This module is shared by the oracle side (tests, CPU baseline) and the HIP
side (tests, benchmark) so that both see the same bytes.  It holds no part
of the method's arithmetic: it only draws random numbers and encodes them
(bf16 by round-to-nearest-even on the raw fp32 bits, gate probabilities as
fp32).  Everything it returns is a plain numpy array.
"""
from .logo_inputs import (  # noqa: F401
    DECODE_WORKLOADS,
    WORKLOADS,
    Workload,
    bf16_bits_from_f32,
    f32_from_bf16_bits,
    make_decode_inputs,
    make_dout,
    make_gate_only,
    make_inputs,
    small_workload,
    markov_burst_gate,
)
