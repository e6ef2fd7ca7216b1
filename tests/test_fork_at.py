"""Fallback inside a segment (treepo_fork_at): the oracle's pins and the
library against the oracle, bit-exact (host only)."""

import numpy as np
import pytest

from oracle import metadata as M
from tests.lib_helpers import host_ctx


def _tree(model_or_ctx, lib):
    """Root 1024 tokens (16 blocks); fork 2 x 1024; fill: root full, children 700 / 1024."""
    if lib:
        r = model_or_ctx.new_root(1024)
        model_or_ctx.kv_commit([r], [1024])
        a, b = model_or_ctx.fork(r, 2, 1024)
        model_or_ctx.kv_commit([a, b], [700, 1024])
        c, = model_or_ctx.fork(b, 1, 512)
        model_or_ctx.kv_commit([c], [300])
    else:
        r = model_or_ctx.new_root(1024)
        model_or_ctx.append([r], [1024])
        a, b = model_or_ctx.fork(r, 2, 1024)
        model_or_ctx.append([a, b], [700, 1024])
        c, = model_or_ctx.fork(b, 1, 512)
        model_or_ctx.append([c], [300])
    return r, a, b, c


def test_split_keeps_every_trajectory():
    """Pins of the oracle's fork_at: each existing leaf keeps exactly its
    block table (the same pool blocks, in order) and token count; depths
    equal chain length - 1; a node starts where its parent ends; ids: the tail, then the children; the children
    start after the kept prefix and share its blocks."""
    m = M.TreeModel(64, 10_000, 10_000)
    r, a, b, c = _tree(m, False)
    leaves = [a, c]
    before = {x: (m.leaf_blocks(x), m.chain_len(x)) for x in leaves}
    n0 = len(m.nodes)
    kids, t = m.fork_at(b, 512, 2, 256)                # split b (1024 tokens) at 512
    assert t == n0 and kids == [n0 + 1, n0 + 2]
    for x in leaves:
        assert (m.leaf_blocks(x), m.chain_len(x)) == before[x]
    for i, nd in enumerate(m.nodes):
        assert nd["depth"] == len(m.chain(i)) - 1
        if nd["parent"] >= 0:                          # a node starts where its parent's tokens end
            p = m.nodes[nd["parent"]]
            assert nd["start"] == p["start"] + p["len"]
    assert m.chain(c) == [r, b, t, c]
    for k in kids:
        assert m.chain(k) == [r, b, k]
        assert m.nodes[k]["start"] == m.nodes[r]["len"] + 512
    # the kept prefix of b: its first 512 tokens = the first 8 blocks of b's old range
    assert m.leaf_blocks(kids[0])[:16 + 8] == before[c][0][:16 + 8]
    # the tail of an active leaf (a: 700 of 1024) keeps growing
    kids2, t2 = m.fork_at(a, 640, 1, 64)
    assert m.nodes[t2]["len"] == 60 and m.nodes[t2]["cap"] == 384
    m.append([t2], [324])
    with pytest.raises(M.TreeError):
        m.append([t2], [1])
    with pytest.raises(M.TreeError):
        m.append([a], [1])                            # the kept prefix is frozen


@pytest.mark.parametrize("offset,n", [(0, 1), (64, 0), (512, 2), (960, 3), (1024, 2)])
def test_library_matches_oracle(offset, n):
    m = M.TreeModel(64, 10_000, 10_000)
    ctx = host_ctx(num_blocks=10_000, max_nodes=10_000)
    _tree(m, False)
    r, a, b, c = _tree(ctx, True)
    got = ctx.fork_at(b, offset, n, 128)
    want = m.fork_at(b, offset, n, 128)
    assert got == want
    ref = np.array([m.record(i) for i in range(len(m.nodes))], dtype=np.int32)
    assert np.array_equal(ctx.export_nodes().reshape(-1, 8), ref)
    # chains and block tables of every node agree
    ids = list(range(len(m.nodes)))
    off, nodes, boff, blocks = ctx.export_chains(ids)[:4]
    for i, x in enumerate(ids):
        assert list(nodes[off[i]:off[i + 1]]) == m.chain(x)
        assert list(blocks[boff[i]:boff[i + 1]]) == m.leaf_blocks(x)


def _fork_at_mutant(kind):
    """fork_at with one plausible mistake planted after the fact."""
    orig = M.TreeModel.fork_at

    def fork_at(self, node, offset, n, cap):
        kids, t = orig(self, node, offset, n, cap)
        if t < 0:
            return kids, t
        tl, x = self.nodes[t], self.nodes[node]
        if kind == "tail_blocks_not_shifted":
            tl["block_begin"] = x["block_begin"]
        elif kind == "tail_len_not_cut":
            x["len"] += tl["len"]
        elif kind == "no_depth_shift":
            for c in range(len(self.nodes)):
                if c != t and t in self.chain(c):
                    self.nodes[c]["depth"] -= 1
        elif kind == "children_not_moved":
            for c in range(len(self.nodes)):
                if self.nodes[c]["parent"] == t:
                    self.nodes[c]["parent"] = node
        elif kind == "tail_starts_at_node":
            tl["start"] = x["start"]
        return kids, t
    return fork_at


@pytest.mark.parametrize("kind", ["tail_blocks_not_shifted", "tail_len_not_cut", "no_depth_shift",
                                  "children_not_moved", "tail_starts_at_node"])
def test_fork_at_mutation_caught(kind, monkeypatch):
    monkeypatch.setattr(M.TreeModel, "fork_at", _fork_at_mutant(kind))
    with pytest.raises(AssertionError):
        test_split_keeps_every_trajectory()
