"""fp64 reference decode attention over segment-tree chains.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The definition (TreePO Sec. 2.3, segment decomposition ``o = s_1 + ... + s_j``
as concatenation; Sec. 2.2 segment-level decoding, where each new token of a
path is decoded against the whole path so far):

* a leaf ``x``'s key/value sequence is the concatenation, root first, of the
  first ``len_n`` rows of every node ``n`` on its chain;
* for query head ``h`` the KV head is ``g = h // G`` with ``G = Hq / Hkv``
  (contiguous groups of query heads share a KV head);
* ``s_t = scale * <q[x, h], K_x[t, g]>``; ``w = softmax(s)``;
  ``out[x, h] = sum_t w_t V_x[t, g]``; ``lse[x, h] = log sum_t exp(s_t)``.

Inputs are bf16 bit patterns, widened exactly to fp64.  Everything is
computed in fp64 with numpy; no blocking, no reordering beyond the definition.
"""

from __future__ import annotations

import numpy as np


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns (uint16) to float64."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


def kv_head(h: int, group: int) -> int:
    """KV head serving query head ``h`` when ``group`` query heads share one."""
    return h // group


def materialize(model, node_kv, x: int, cache: dict | None = None):
    """K_x, V_x of leaf ``x``: its chain's rows concatenated, fp64 [L, Hkv, D].

    ``node_kv(n)`` returns the (K bits, V bits) rows of node ``n``; only the
    first ``len_n`` rows are used.
    """
    ks, vs = [], []
    for n in model.chain(x):
        ln = model.nodes[n]["len"]
        if cache is not None and n in cache:
            k, v = cache[n]
        else:
            kb, vb = node_kv(n)
            k, v = bf16_bits_to_f64(kb[:ln]), bf16_bits_to_f64(vb[:ln])
            if cache is not None:
                cache[n] = (k, v)
        ks.append(k)
        vs.append(v)
    return np.concatenate(ks, axis=0), np.concatenate(vs, axis=0)


def attend(q: np.ndarray, K: np.ndarray, V: np.ndarray, scale: float):
    """Textbook softmax attention of one decode position.

    q: [Hq, D]; K, V: [L, Hkv, D] (fp64).  Returns out [Hq, D], lse [Hq].
    """
    hq = q.shape[0]
    hkv = K.shape[1]
    group = hq // hkv
    out = np.empty((hq, V.shape[2]), dtype=np.float64)
    lse = np.empty(hq, dtype=np.float64)
    for h in range(hq):
        g = kv_head(h, group)
        s = scale * (K[:, g, :] @ q[h])
        m = s.max()
        e = np.exp(s - m)
        z = e.sum()
        out[h] = (e @ V[:, g, :]) / z
        lse[h] = m + np.log(z)
    return out, lse


def tree_decode(model, node_kv, leaves, q_bits: np.ndarray, scale: float,
                positions=None):
    """Reference outputs for a decode call.

    ``q_bits`` is [n_leaves, Hq, D] (bf16 bits) in call order.  ``positions``
    restricts the work to some call positions (for sampled checks of large
    workloads); the returned arrays then hold only those rows, in that order.
    """
    model.check_decode(leaves)
    pos = range(len(leaves)) if positions is None else positions
    cache: dict = {}
    outs, lses = [], []
    for p in pos:
        K, V = materialize(model, node_kv, leaves[p], cache)
        o, l = attend(bf16_bits_to_f64(q_bits[p]), K, V, scale)
        outs.append(o)
        lses.append(l)
    return np.stack(outs), np.stack(lses)
