"""Pins of the fp64 TreePO advantage oracle (oracle/advantage.py).

Each pin checks the oracle against something other than its own formula: a
hand-worked example (Sec. 2.3, Fig. 3 tree), the GRPO advantage that a
depth-1 tree reduces to, and invariants that the definition implies
(rejection, one global std, affine reward maps, zero-sum sub-groups).
Every pin raises AssertionError on a mismatch.
"""

from __future__ import annotations

import os

import numpy as np

from oracle import advantage as ADV

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "advantage_fig3.txt")


def fig3_tree():
    """Parents of the Fig. 3 tree: q=0; c=1, c'=2; c1..c4=3..6; leaves 7..14."""
    parents = [-1, 0, 0, 1, 1, 2, 2] + [3, 3, 4, 4, 5, 5, 6, 6]
    return parents, list(range(7, 15))


def pin_fig3_golden(tol=1e-12):
    parents, leaves = fig3_tree()
    rows = [ln.split() for ln in open(GOLDEN) if ln.strip() and not ln.startswith("#")]
    R = [float(r[1]) for r in rows]
    mean_w = np.array([float(r[2]) for r in rows])
    size_w = np.array([float(r[3]) for r in rows])
    assert np.abs(ADV.tree_advantage(parents, leaves, R, "mean") - mean_w).max() <= tol
    assert np.abs(ADV.tree_advantage(parents, leaves, R, "size") - size_w).max() <= tol


def pin_depth1_is_grpo(seeds=(1, 2, 3), tol=1e-12):
    """A root with n leaf children: one sub-group (the query), so both
    aggregations give the GRPO advantage (R - mean R) / std R (population)."""
    for seed in seeds:
        rng = np.random.default_rng(seed)
        n = int(rng.integers(2, 20))
        R = rng.normal(size=n)
        parents = [-1] + [0] * n
        want = (R - R.mean()) / R.std()
        for w in ("mean", "size"):
            assert np.abs(ADV.tree_advantage(parents, list(range(1, n + 1)), R, w) - want).max() <= tol


def random_forest(seed, n_roots=3, max_children=3, depth=4):
    """Random forest (parents list) and its leaves, every node forking 1..max_children."""
    rng = np.random.default_rng(seed)
    parents, frontier = [], []
    for _ in range(n_roots):
        parents.append(-1)
        frontier.append(len(parents) - 1)
    for _ in range(depth):
        nxt = []
        for x in frontier:
            for _ in range(int(rng.integers(1, max_children + 1))):
                parents.append(x)
                nxt.append(len(parents) - 1)
        frontier = nxt
    return parents, frontier


def pin_rejection(tol=1e-12):
    """A query whose trajectories share one reward gets 0 and leaves the
    other queries' advantages as they are alone."""
    parents, leaves = random_forest(7, n_roots=2)
    chains = [ADV.chain(parents, x) for x in leaves]
    rng = np.random.default_rng(8)
    R = rng.integers(0, 2, size=len(leaves)).astype(float)
    first = np.array([c[0] == chains[0][0] for c in chains])
    R[~first] = 1.0  # the second query: all equal
    R[np.flatnonzero(first)[0]] = 1.0 - R[np.flatnonzero(first)[1]]  # the first query is not all equal
    both = ADV.tree_advantage(parents, leaves, R)
    assert np.all(both[~first] == 0.0)
    alone = ADV.tree_advantage(parents, [x for x, f in zip(leaves, first) if f], R[first])
    assert np.abs(both[first] - alone).max() <= tol
    assert np.abs(alone).max() > 0.1


def pin_global_std(tol=1e-12):
    """Two copies of one query, the second with rewards doubled: every
    sub-group advantage of the copy doubles, so the global variance is
    (1 + 4) / 2 times the first query's, and the first query's advantages in
    the batch are its advantages alone divided by sqrt(2.5)."""
    parents, leaves = fig3_tree()
    R = np.array([1, 0, 1, 1, 0, 0, 0, 1], dtype=float)
    off = len(parents)
    parents2 = parents + [p + off if p >= 0 else -1 for p in parents]
    leaves2 = leaves + [x + off for x in leaves]
    R2 = np.concatenate([R, 2 * R])
    alone = ADV.tree_advantage(parents, leaves, R)
    batch = ADV.tree_advantage(parents2, leaves2, R2)
    assert np.abs(batch[:8] - alone / np.sqrt(2.5)).max() <= tol
    assert np.abs(batch[8:] - 2 * alone / np.sqrt(2.5)).max() <= tol


def pin_affine_invariance(seeds=(11, 12), tol=1e-10):
    """R -> a R + b (a > 0, the same for the whole batch) leaves the advantages unchanged."""
    for seed in seeds:
        parents, leaves = random_forest(seed)
        R = np.random.default_rng(seed).normal(size=len(leaves))
        for w in ("mean", "size"):
            a0 = ADV.tree_advantage(parents, leaves, R, w)
            a1 = ADV.tree_advantage(parents, leaves, 3.5 * R - 2.0, w)
            assert np.abs(a0 - a1).max() <= tol


def pin_zero_sum_subgroups(seeds=(21, 22), tol=1e-12):
    """Each sub-group's advantages are deviations from its mean: they sum to 0
    over its members, and the predecessors of a leaf are its chain minus
    itself."""
    for seed in seeds:
        parents, leaves = random_forest(seed)
        R = np.random.default_rng(seed).normal(size=len(leaves))
        rows, chains = ADV.subgroup_advantages(parents, leaves, R)
        per = {}
        for p, row in enumerate(rows):
            assert [a for (a, _, _) in row] == chains[p][:-1]
            for (a, size, x) in row:
                per.setdefault(a, []).append(x)
                assert size == sum(1 for c in chains if a in c)
        for a, xs in per.items():
            assert abs(sum(xs)) <= tol * max(1, len(xs))


def pin_duplicates(tol=0.0):
    """The same leaf at two call positions (two identical trajectories) gets
    the same advantage."""
    parents, leaves = fig3_tree()
    lv = leaves + [leaves[2]]
    R = [1, 0, 1, 1, 0, 0, 0, 1, 1]
    adv = ADV.tree_advantage(parents, lv, R)
    assert abs(adv[2] - adv[8]) <= tol


ALL = [pin_fig3_golden, pin_depth1_is_grpo, pin_rejection, pin_global_std, pin_affine_invariance,
       pin_zero_sum_subgroups, pin_duplicates]
