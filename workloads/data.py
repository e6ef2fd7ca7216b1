"""Seeded bf16 input data.

Every random stream is a numpy ``Generator(PCG64)`` seeded from
``SeedSequence([config_seed, kind, index])``.  Node K/V rows are keyed by the
node id, so any node can be regenerated on its own (the oracle never has to
hold a whole 11.8 GB pool); queries are keyed by the decode-step index.

Values are drawn as fp32 standard normals and rounded to bf16 with
round-to-nearest-even on the fp32 bit pattern.  The result is returned as the
raw ``uint16`` bit patterns; consumers decide how to widen them.
"""

from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

KIND_K = 1
KIND_V = 2
KIND_Q = 3
KIND_STRUCT = 4


def _rng(seed: int, kind: int, index: int) -> np.random.Generator:
    return np.random.Generator(
        np.random.PCG64(np.random.SeedSequence([int(seed), int(kind), int(index)])))


def bf16_round_bits(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns, round-to-nearest-even (finite inputs)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    return ((u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)).astype(np.uint16)


def normal_bits(seed: int, kind: int, index: int, shape) -> np.ndarray:
    x = _rng(seed, kind, index).standard_normal(shape, dtype=np.float32)
    return bf16_round_bits(x)


def node_kv_bits(seed: int, node: int, rows: int, hkv: int, d: int):
    """K and V bit patterns for rows ``[0, rows)`` of a node, shape [rows, Hkv, D].

    Row ``r`` is the node's ``r``-th token; a node's stream is fixed by
    (seed, node), so rows appended in several calls come from one stream.
    """
    k = normal_bits(seed, KIND_K, node, (rows, hkv, d))
    v = normal_bits(seed, KIND_V, node, (rows, hkv, d))
    return k, v


def many_node_kv_bits(seed: int, nodes_rows, hkv: int, d: int, threads: int | None = None):
    """``node_kv_bits`` for many (node, rows) pairs, generated on a thread pool."""
    threads = threads or min(16, os.cpu_count() or 1)
    with ThreadPoolExecutor(threads) as ex:
        return list(ex.map(lambda nr: node_kv_bits(seed, nr[0], nr[1], hkv, d), nodes_rows))


def query_bits(seed: int, step: int, n_leaves: int, hq: int, d: int) -> np.ndarray:
    """Decode-step query bit patterns, shape [n_leaves, Hq, D]."""
    return normal_bits(seed, KIND_Q, step, (n_leaves, hq, d))


def structure_rng(seed: int) -> np.random.Generator:
    """Stream for the tree-shape draws of the randomised configs."""
    return _rng(seed, KIND_STRUCT, 0)
