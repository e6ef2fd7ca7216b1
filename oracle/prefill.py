"""fp64 reference prefill: causal attention of newly appended tokens
(TEST INFRASTRUCTURE ONLY; see the package docstring).

The shared prompt of a query is the root of its tree; it is prefilled once
and its K/V serve every rollout of the query (Sec. 2.2 tree rollout; the
shared-prefix prefilling of the sampling-efficiency analysis, Sec. 4.1).  The
definition, for tokens appended to node ``x`` (the model holds the state
*after* the append): a new token at chain position ``p`` (``p`` counts the
tokens of ``x``'s chain before it, root first) attends with textbook softmax
to chain positions ``0..p`` -- every earlier token of its chain and itself --
with the same head map and scale as decode:
``out[p, h] = sum_{t <= p} softmax_t(scale <q_p,h, K[t, g]>) V[t, g]`` and
``lse[p, h] = log sum_{t <= p} exp(scale <q_p,h, K[t, g]>)``.
"""

from __future__ import annotations

import numpy as np

from .attention import attend, bf16_bits_to_f64, materialize


def prefill(model, node_kv, nodes, ntok, q_bits: np.ndarray, scale: float, rows=None):
    """Reference outputs of a prefill call.

    ``nodes[i]`` received its last ``ntok[i]`` tokens in this call; ``q_bits``
    is [sum ntok, Hq, D] (bf16 bits) packed in call order.  ``rows`` restricts
    the work to some packed rows (sampled checks).  Returns out [R, Hq, D],
    lse [R, Hq] for the selected rows, in order.
    """
    want = None if rows is None else set(int(r) for r in rows)
    outs, lses = {}, {}
    base = 0
    for x, n in zip(nodes, ntok):
        if n and (want is None or any(base <= r < base + n for r in want)):
            K, V = materialize(model, node_kv, x)
            first = K.shape[0] - n
            for j in range(n):
                r = base + j
                if want is not None and r not in want:
                    continue
                p = first + j
                outs[r], lses[r] = attend(bf16_bits_to_f64(q_bits[r]), K[:p + 1], V[:p + 1], scale)
        base += n
    order = sorted(outs) if rows is None else [int(r) for r in rows]
    hq, d = q_bits.shape[1], q_bits.shape[2]
    if not order:
        return np.zeros((0, hq, d)), np.zeros((0, hq))
    return np.stack([outs[r] for r in order]), np.stack([lses[r] for r in order])
