"""Log-sum-exp algebra for merging per-node partial attention (fp64).

TEST INFRASTRUCTURE ONLY (see the package docstring).

Splitting a leaf's concatenated sequence into pieces (its chain's segments, or
token chunks of them) and scoring each piece separately gives, per piece ``i``
and query head, a partial ``(O_i, m_i, l_i)``:

* ``m_i = max_t s_t`` over the piece (``-inf`` for an empty piece),
* ``l_i = sum_t exp(s_t - m_i)``,
* ``O_i = sum_t exp(s_t - m_i) V_t`` (unnormalised).

With ``m* = max_i m_i`` and ``L = sum_i l_i exp(m_i - m*)`` the merged result
is ``out = sum_i exp(m_i - m*) O_i / L`` and ``lse = m* + log L``.  This equals
the direct softmax over the whole sequence, which is why sharing an ancestor's
KV across all of its descendant leaves (TreePO Sec. 2.1, shared prefixes
represented once) cannot change the answer.  Empty pieces contribute nothing.
"""

from __future__ import annotations

import numpy as np


def partial(q: np.ndarray, K: np.ndarray, V: np.ndarray, scale: float):
    """Partial of one piece for one head: q [D], K/V [T, D] -> (O [D], m, l)."""
    if K.shape[0] == 0:
        return np.zeros(V.shape[1]), -np.inf, 0.0
    s = scale * (K @ q)
    m = s.max()
    e = np.exp(s - m)
    return e @ V, m, e.sum()


def combine(parts):
    """Merge partials ``[(O, m, l), ...]`` -> (out [D], lse)."""
    ms = np.array([p[1] for p in parts], dtype=np.float64)
    m_star = ms.max()
    if m_star == -np.inf:
        raise ValueError("all pieces empty")
    w = np.exp(ms - m_star)
    L = sum(wi * p[2] for wi, p in zip(w, parts))
    O = sum(wi * p[0] for wi, p in zip(w, parts))
    return O / L, m_star + np.log(L)
