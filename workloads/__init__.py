"""Seeded synthetic workloads for segment-tree decode attention.

This package only *generates inputs*: tree-building call logs shaped like
TreePO rollouts (Alg. 1, segment-level tree sampling in Sec. 2.2) and the
bf16 bit patterns of the per-node K/V rows and per-leaf queries.  It holds
none of the attention arithmetic; both the fp64 oracle and the GPU harness
consume what it produces.
"""

from .data import (KIND_K, KIND_V, KIND_Q, KIND_STRUCT, bf16_round_bits,
                   node_kv_bits, query_bits, structure_rng)
from .configs import CONFIGS, Config, CallLog, build_call_log

__all__ = [
    "KIND_K", "KIND_V", "KIND_Q", "KIND_STRUCT", "bf16_round_bits",
    "node_kv_bits", "query_bits", "structure_rng", "CONFIGS", "Config",
    "CallLog", "build_call_log",
]
