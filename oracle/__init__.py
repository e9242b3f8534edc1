"""CPU oracle for one UniF-MoE feed-forward layer (test infrastructure only).

Only tests, the smoke check and the benchmark's CPU-baseline leg may import
this package; the HIP library never does and has no fallback to it.
"""
from .unif_moe_oracle import (  # noqa: F401
    route, forward, forced_forward, margins, stats, decisions, gelu,
    shared_offset, block_count, ExpertWeights,
)
