"""Structural fixtures taken from the paper's worked example."""

import os

from oracle import metadata as M
from workloads import build_call_log

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _read(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append([int(x) for x in line.split()])
    return rows


def test_fig3_subgroups_match_tiny_tree():
    """The 8-leaf, depth-3 binary tree of Fig. 3 is config 1's shape: its
    node->descendant-leaf sets are the nested sub-groups of Eq. (groups)."""
    log = build_call_log(1)
    m = M.replay(log, 64, 1000, 1000)
    ds = m.desc_sets(log.leaves)
    for depth, size, count in _read("fig3_subgroups.txt"):
        sets = [v for n, v in ds.items() if m.nodes[n]["depth"] == depth]
        assert len(sets) == count
        assert all(len(s) == size for s in sets)
    # nesting: every leaf's sub-groups shrink along its chain
    for pos, x in enumerate(log.leaves):
        sizes = [len(ds[n]) for n in m.chain(x)]
        assert sizes == [8, 4, 2, 1]
        for a, b in zip(m.chain(x), m.chain(x)[1:]):
            assert set(ds[b]) <= set(ds[a]) and pos in ds[b]
