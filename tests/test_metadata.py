"""Library node table, chains, block tables and descendant sets vs the oracle
model, bit-exact (int32 equality), on all five workloads and random trees."""

import numpy as np
import pytest

from oracle import metadata as M
from tests.lib_helpers import host_ctx, oracle_model, replay_host
from tests.oracle_pins import random_tiny_tree, _Log
from workloads import build_call_log


def _compare(ctx, model, leaves):
    rec = ctx.export_nodes()
    ref = np.array([model.record(n) for n in range(len(model.nodes))], dtype=np.int32)
    assert rec.shape == ref.shape and np.array_equal(rec, ref)
    co, cn, bo, bl = ctx.export_chains(leaves)
    rco, rcn, rbo, rbl = [0], [], [0], []
    for x in leaves:
        rcn += model.chain(x); rco.append(len(rcn))
        rbl += model.leaf_blocks(x); rbo.append(len(rbl))
    assert np.array_equal(co, rco) and np.array_equal(cn, rcn)
    assert np.array_equal(bo, rbo) and np.array_equal(bl, rbl)
    nodes, off, desc = ctx.export_desc(leaves)
    ds = model.desc_sets(leaves)
    assert list(nodes) == list(ds.keys())
    assert np.array_equal(desc, [p for v in ds.values() for p in v])
    assert np.array_equal(np.diff(off), [len(v) for v in ds.values()])


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_workload_metadata_bit_exact(cfg):
    log = build_call_log(cfg)
    ctx = host_ctx()
    ids = replay_host(ctx, log)
    assert ids == list(range(log.n_nodes))
    _compare(ctx, oracle_model(log), log.leaves)


@pytest.mark.parametrize("seed", range(40))
def test_random_tree_metadata_bit_exact(seed):
    ops, leaves, rows, _ = random_tiny_tree(seed, max_leaves=12, max_tokens=700)
    log = _Log(ops, leaves, rows)
    ctx = host_ctx()
    replay_host(ctx, log)
    model = oracle_model(log)
    _compare(ctx, model, leaves or [0])


def test_kv_slots_follow_block_reservation():
    ctx = host_ctx()
    r = ctx.new_root(100)            # blocks 0, 1
    a, b = ctx.fork(r, 2, 70)        # blocks 2-3, 4-5
    rows = ctx.kv_slots([a, b, a], [3, 2, 65])
    assert list(rows[:3]) == [128, 129, 130]
    assert list(rows[3:5]) == [256, 257]
    assert list(rows[5:]) == list(range(131, 196))
    ctx.kv_commit([a], [10])
    assert list(ctx.kv_slots([a], [2])) == [138, 139]


def _plan_checks(ctx, model, leaves, mode):
    items, rowsets, tiles = ctx.export_plan(leaves, mode)
    G = ctx.cfg.num_q_heads // ctx.cfg.num_kv_heads
    covered = {x: [] for x in range(len(leaves))}
    for it in items:
        kind, rb, nl, tb, te, pbase, rows, run = it[:8]
        assert rows == nl * G and te > tb and nl >= 1
        for f in range(3):   # the first tiles' half-block sources ride in the record
            want_src = 2 * tiles[tb + f][0] + (tiles[tb + f][2] & 1) if tb + f < te else -1
            assert it[8 + f] == want_src
        for pos in rowsets[rb:rb + nl]:
            for t in tiles[tb:te]:
                covered[pos].append(tuple(t))
    for pos, x in enumerate(leaves):
        got = sorted(covered[pos])
        want = []
        for n in model.chain(x):
            ln = model.nodes[n]["len"]
            for k in range((ln + 31) // 32):     # 32-token tiles, two per 64-token block
                want.append((model.nodes[n]["block_begin"] + k // 2, n, k, min(32, ln - 32 * k)))
        assert got == sorted(want), (mode, pos)
    # partial rows are laid out back to back without overlap
    bases = sorted((it[5], it[6] * ctx.cfg.num_kv_heads) for it in items)
    for (b0, s0), (b1, _) in zip(bases, bases[1:]):
        assert b0 + s0 == b1
    return items, tiles


@pytest.mark.parametrize("cfg", [1, 2, 4])
def test_plan_covers_each_chain_token_once(cfg):
    log = build_call_log(cfg)
    from workloads import CONFIGS
    c = CONFIGS[cfg]
    ctx = host_ctx(hq=c.hq, hkv=c.hkv, d=c.d)
    replay_host(ctx, log)
    model = oracle_model(log)
    items_t, tiles_t = _plan_checks(ctx, model, log.leaves, 0)
    items_n, tiles_n = _plan_checks(ctx, model, log.leaves, 1)
    # the tree plan streams every node once per leaf group; the naive plan once per leaf
    tree_tok = sum(int(t[3]) for it in items_t for t in tiles_t[it[3]:it[4]])
    naive_tok = sum(int(t[3]) for it in items_n for t in tiles_n[it[3]:it[4]])
    logical = sum(model.chain_len(x) for x in log.leaves)
    assert naive_tok == logical
    assert tree_tok <= naive_tok


def test_duplicate_and_interior_leaves():
    ctx = host_ctx()
    r = ctx.new_root(64); ctx.kv_commit([r], [10])
    a, b = ctx.fork(r, 2, 64); ctx.kv_commit([a, b], [5, 0])
    leaves = [a, r, a, b]          # interior node, duplicate, zero-length leaf
    log = _Log([("root", 64), ("append", [r], [10]), ("fork", r, 2, 64), ("append", [a, b], [5, 0])],
               leaves, {r: 10, a: 5, b: 0})
    model = oracle_model(log)
    _compare(ctx, model, leaves)
    _plan_checks(ctx, model, leaves, 0)


def test_schedule_option_sets_item_kinds():
    """VALU_MAX_ROWS moves items between the shuffle and MFMA partials; the
    plan's coverage is unchanged and out-of-range values are rejected."""
    from paper_2508_17445_amd import OPT_VALU_MAX_ROWS, TreePOError
    from workloads import CONFIGS
    log = build_call_log(2)
    c = CONFIGS[2]
    ctx = host_ctx(hq=c.hq, hkv=c.hkv, d=c.d)
    replay_host(ctx, log)
    model = oracle_model(log)
    kinds = {}
    for v in (0, 8):
        ctx.set_option(OPT_VALU_MAX_ROWS, v)
        assert ctx.get_option(OPT_VALU_MAX_ROWS) == v
        items, _ = _plan_checks(ctx, model, log.leaves, 0)
        kinds[v] = items[:, 0]
        if v == 0:
            assert (items[:, 0] == 1).all()
        else:
            # VALU items are exactly those of at most 8 rows, and come first
            assert ((items[:, 0] == 0) == (items[:, 6] <= 8)).all()
            assert (np.diff(items[:, 0]) >= 0).all()
    assert (kinds[8] == 0).any()
    for bad in (-1, 9):
        with pytest.raises(TreePOError):
            ctx.set_option(OPT_VALU_MAX_ROWS, bad)
    with pytest.raises(TreePOError):
        ctx.set_option(12345, 0)
