"""TreePO advantage over the rollout tree, fp64 (TEST INFRASTRUCTURE ONLY).

Nothing in the product path may import this module; it shares no code with
the HIP library.  It follows TreePO Sec. 2.3 (Eq. groups, Eq. tree_ae) and
the size-weighted variant of Sec. 4.2 (Eq. tree_ae_sgw), taking the steps in
the paper's order:

1. A trajectory is a decoded leaf (one call position p, node leaves[p]); its
   segments are the nodes of its root-to-leaf chain.  A query is a root; its
   group G is every trajectory under that root.
2. Sub-groups (Eq. groups): for each strict predecessor a of the leaf (root
   first, the leaf's own node excluded), G_a = the trajectories whose chain
   contains a.  These are nested: G_{a_d} within ... within G_{a_0} = G.
   (Fig. 3 caption: the sub-groups of a leaf are defined by its
   predecessors.)
3. Sub-group advantage: A_{p,a} = R_p - mean of R over G_a.
4. Aggregation: the plain mean over the leaf's predecessors (Eq. tree_ae),
   or the |G_a|-weighted mean (Eq. tree_ae_sgw).
5. Normalisation by one global standard deviation (the REINFORCE++-style
   global variance normalisation the text names): the population standard
   deviation of every A_{p,a} of every kept query.
6. Dynamic rejection (the constraint that the std of R over G is not zero):
   a query whose trajectories all have the same reward is dropped; its
   trajectories get advantage 0 and add nothing to step 5.

Readings of what the paper leaves open: the
garbled `std(...)^{J-1}` term is read as step 5; a leaf with no predecessor
(a root decoded as a trajectory) gets 0; if no query is kept or the global
std is 0, every advantage is 0.
"""

from __future__ import annotations

import numpy as np


def chain(parents, x: int) -> list[int]:
    """Root-first chain of node x (parents[root] < 0)."""
    c = []
    while x >= 0:
        c.append(x)
        x = parents[x]
    return c[::-1]


def subgroup_advantages(parents, leaves, rewards):
    """Per position p: list of (predecessor node a, |G_a|, A_{p,a}), root first."""
    chains = [chain(parents, int(x)) for x in leaves]
    members: dict[int, list[int]] = {}
    for p, ch in enumerate(chains):
        for a in ch:
            members.setdefault(a, []).append(p)
    R = np.asarray(rewards, dtype=np.float64)
    rows = []
    for p, ch in enumerate(chains):
        row = []
        for a in ch[:-1]:
            g = members[a]
            row.append((a, len(g), R[p] - R[g].mean()))
        rows.append(row)
    return rows, chains


def tree_advantage(parents, leaves, rewards, weighting: str = "mean"):
    """Advantage per call position (fp64).  weighting: "mean" (Eq. tree_ae)
    or "size" (Eq. tree_ae_sgw)."""
    if weighting not in ("mean", "size"):
        raise ValueError(weighting)
    R = np.asarray(rewards, dtype=np.float64)
    n = len(leaves)
    rows, chains = subgroup_advantages(parents, leaves, rewards)
    roots = [ch[0] for ch in chains]
    kept_root = {}
    for r in set(roots):
        g = [p for p in range(n) if roots[p] == r]
        kept_root[r] = bool(np.std(R[g]) != 0.0)
    kept = [kept_root[roots[p]] for p in range(n)]
    pairs = [a for p in range(n) if kept[p] for (_, _, a) in rows[p]]
    adv = np.zeros(n, dtype=np.float64)
    if not pairs:
        return adv
    sigma = float(np.std(np.asarray(pairs)))
    if sigma == 0.0:
        return adv
    for p in range(n):
        if not kept[p] or not rows[p]:
            continue
        a = np.array([x for (_, _, x) in rows[p]])
        if weighting == "mean":
            pooled = a.mean()
        else:
            w = np.array([s for (_, s, _) in rows[p]], dtype=np.float64)
            pooled = (w * a).sum() / w.sum()
        adv[p] = pooled / sigma
    return adv


def from_model(model, leaves, rewards, weighting: str = "mean"):
    """tree_advantage over an oracle metadata model (oracle.metadata.TreeModel)."""
    parents = [nd["parent"] for nd in model.nodes]
    return tree_advantage(parents, leaves, rewards, weighting)
