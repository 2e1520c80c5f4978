"""Seeded synthetic inputs shared by the oracle side and the HIP side.

This package holds random-number synthesis and workload shapes only: no
dequantisation, no linear algebra, no routing.  Both the CPU oracle tests and
the GPU path draw their inputs from here, so a parity comparison always sees
identical bytes on both sides.
"""
from .gen import (  # noqa: F401
    stream_key, words, uniform01, normal, to_f16,
    int4_codes, group_scales, activations, exact_activations, sign_activations, exact_scales,
    router_weights, permutation, scores,
)
