"""Seeded synthetic inputs shared by the oracle tests, the GPU tests and the bench.

This package holds workload definitions (shapes, partition offsets, the fixed
selection masks of the sweep workloads) and the random tensors that stand in for
video-DiT activations.  It contains none of the method's arithmetic: no
attention, no state merge, no weights.  Both sides of every parity check take
their inputs from here and from nowhere else.
"""
from .workloads import WORKLOADS, Workload, get_workload  # noqa: F401
from .gen import (  # noqa: F401
    bf16_round,
    bf16_bits,
    gen_qkv,
    query_block,
    gen_evolved,
    sample_rows,
)
