"""Seeded synthetic workloads for the mixed-bit linear layer.

This package only *generates inputs*: activations, weights, the channel
ranking, the block lengths, the channel permutation and the group-quantized
codes with their fp16 scales and zero points.  It holds none of the arithmetic
of the hot path (no dequantization, no matrix product); both the oracle and the
HIP library consume what it produces.
"""
from .workloads import *  # noqa: F401,F403
