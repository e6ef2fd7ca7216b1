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


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5, 6])
@pytest.mark.parametrize("bt", [16, 32, 64])
def test_workload_metadata_bit_exact(cfg, bt):
    log = build_call_log(cfg)
    ctx = host_ctx(block_tokens=bt)
    ids = replay_host(ctx, log)
    assert ids == list(range(log.n_nodes))
    _compare(ctx, oracle_model(log, block_tokens=bt), log.leaves)


@pytest.mark.parametrize("seed", range(40))
def test_random_tree_metadata_bit_exact(seed):
    ops, leaves, rows, _ = random_tiny_tree(seed, max_leaves=12, max_tokens=700)
    log = _Log(ops, leaves, rows)
    bt = (16, 32, 64)[seed % 3]
    ctx = host_ctx(block_tokens=bt)
    replay_host(ctx, log)
    model = oracle_model(log, block_tokens=bt)
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


MAX_STREAM_TILES = 256
MAX_BLOCK_INTS = 4 + 4 * 128 + 2 * 256 + 2 * 256 + 2 * 256   # header, pieces, tiles, segments, dests, live


def _tile_cost(rows):
    return 1.0 if rows <= 16 else 1.1 if rows <= 32 else 1.4 if rows <= 64 else 2.6


# planner speeds: second workgroup slot of a CU, and the odd-numbered XCDs
# (stream s runs on XCD s % 8)
SLOT1_SPEED, ODD_XCD_SPEED = 0.80, 0.935


def _speed(s, cus=256, xcds=8):
    s = np.asarray(s)
    odd = (s % xcds) % 2 == 1 if xcds > 1 else np.zeros(s.shape, bool)
    return np.where(s < cus, 1.0, SLOT1_SPEED) * np.where(odd, ODD_XCD_SPEED, 1.0)


def _plan_checks(ctx, model, leaves, mode):
    pieces, rowsets, tiles, n_streams = ctx.export_plan(leaves, mode)
    hkv = ctx.cfg.num_kv_heads
    G = ctx.cfg.num_q_heads // hkv
    covered = {(x, g): [] for x in range(len(leaves)) for g in range(hkv)}
    stream_next = {}
    seg_next = {}
    for pc in pieces:
        rb, nl, rows, g, stile, nt, reserved, seg, run, stream, ptile, nq = pc[:12]
        assert rows == nl * G and nt >= 1 and nl >= 1 and 0 <= g < hkv and rows <= 128 and reserved == 0
        assert 0 <= stream < n_streams and (pc[12:] == 0).all()
        assert nq == -(-rows // 64)          # 64 query rows per query tile
        # pieces of a stream are consecutive and tile its list from 0:
        # the piece's query tiles, then its KV tiles
        assert stile == stream_next.get(stream, 0)
        stream_next[stream] = stile + nq + nt
        assert stile + nq + nt <= MAX_STREAM_TILES
        assert seg == seg_next.get(stream, 0)
        seg_next[stream] = seg + nl
        assert seg + nl <= 256
        for pos in rowsets[rb:rb + nl]:
            for t in tiles[ptile:ptile + nt]:
                covered[(pos, g)].append(tuple(t))
    assert sorted(stream_next) == list(range(n_streams))
    live_mode = ctx.cfg.node_len is not None
    for pos, x in enumerate(leaves):
        want = []
        for n in model.chain(x):
            ln, cap = model.nodes[n]["len"], model.nodes[n]["cap"]
            # with device lengths an unfrozen node is covered up to its capacity
            span = cap if live_mode and model.n_children[n] == 0 and ln < cap else ln
            for k in range((span + 31) // 32):     # 32-token tiles; a tile starts in block 32 k / B
                want.append((model.nodes[n]["block_begin"] + 32 * k // model.B, n, k, max(0, min(32, ln - 32 * k))))
        for g in range(hkv):
            got = sorted(covered[(pos, g)])
            # a reused live plan reports the counts of its planning time (the
            # device reads the current ones): compare those of full tiles only
            assert [t[:3] for t in got] == [t[:3] for t in sorted(want)], (mode, pos, g)
            assert all(a[3] == b[3] or (live_mode and a[3] < b[3]) for a, b in zip(got, sorted(want))), (mode, pos, g)
    _block_checks(ctx, leaves, mode, pieces, rowsets, tiles, n_streams, stream_next, seg_next)
    return pieces, tiles, n_streams


def _block_checks(ctx, leaves, mode, pieces, rowsets, tiles, n_streams, stream_next, seg_next):
    """The kernel's stream blocks restate the exported schedule exactly, every
    pool and query address they lead to is in bounds, and the partial slots
    give each (leaf, KV head) key entries 0..count-1 in piece order."""
    blocks = ctx.export_blocks(leaves, mode)
    hq, hkv, d, nb = ctx.cfg.num_q_heads, ctx.cfg.num_kv_heads, ctx.cfg.head_dim, ctx.cfg.num_blocks
    B = ctx.cfg.block_tokens
    G = hq // hkv
    bi = blocks.shape[1]
    assert blocks.shape[0] == n_streams and bi % 4 == 0 and bi <= MAX_BLOCK_INTS
    by_stream = {}
    count = {}
    for pc in pieces:
        by_stream.setdefault(int(pc[9]), []).append(pc)
        for x in rowsets[pc[0]:pc[0] + pc[1]]:
            count[(int(x), int(pc[3]))] = count.get((int(x), int(pc[3])), 0) + 1
    assert sorted(count) == [(x, g) for x in range(len(leaves)) for g in range(hkv)]
    emax = max(count.values())
    # partial-slot layout: strided (key k at entry k * emax) when the
    # combine's speculative first round reads at most 8 MiB, else compact
    # (prefix sums of the counts, in key order)
    nkeys = len(leaves) * hkv
    spec = nkeys * G * min(emax, 32) * (d * 4 + 8)
    base, acc = {}, 0
    for x in range(len(leaves)):
        for g in range(hkv):
            base[(x, g)] = acc if spec > 8 << 20 else (x * hkv + g) * emax
            acc += count[(x, g)]
    entry = {}
    nodes = ctx.export_nodes()
    kids = np.bincount(nodes[:, 0][nodes[:, 0] >= 0], minlength=len(nodes))
    live_mode = ctx.cfg.node_len is not None
    for s in range(n_streams):
        b = blocks[s]
        n_p, n_t, n_s, n_l = int(b[0]), int(b[1]), int(b[2]), int(b[3])
        pcs = by_stream[s]
        assert (n_p, n_t, n_s) == (len(pcs), stream_next[s], seg_next[s])
        assert live_mode or n_l == 0
        tiles_at = 4 + 4 * n_p
        segs_at = tiles_at + 2 * (n_t + n_t % 2)
        dests_at = segs_at + n_s + (-n_s) % 4
        live_at = dests_at + n_s + (-n_s) % 4
        assert live_at + 2 * n_l <= bi
        assert (b[tiles_at + 2 * n_t:segs_at] == 0).all() and (b[segs_at + n_s:dests_at] == 0).all()
        assert (b[dests_at + n_s:live_at] == 0).all() and (b[live_at + 2 * n_l:] == 0).all()
        recs = b[4:tiles_at].reshape(-1, 4)
        st = b[tiles_at:tiles_at + 2 * n_t].reshape(-1, 2)
        sg = b[segs_at:segs_at + n_s]
        dst = b[dests_at:dests_at + n_s]
        live = b[live_at:live_at + 2 * n_l].reshape(-1, 2)
        used_live = set()
        for i, pc in enumerate(pcs):
            rb, nl, rows, g, stile, nt, _, seg, _, _, ptile, nq = (int(v) for v in pc[:12])
            assert tuple(recs[i]) == (rows, stile, nt, seg)
            for t in range(nq):
                assert tuple(st[stile + t]) == (-1 - seg, (64 * t) | (min(64, rows - 64 * t) << 16))
            for t in range(nt):
                blk, node, tin, valid = (int(v) for v in tiles[ptile + t])
                hb, v = (int(x) for x in st[stile + nq + t])
                # first pool row of the tile over 16, KV head g's rows included
                assert hb * 16 == (g * nb + int(nodes[node][5])) * B + 32 * tin
                assert blk == int(nodes[node][5]) + 32 * tin // B
                assert 0 <= hb and hb * 16 + 32 <= hkv * nb * B
                # a tile of an unfrozen node that was not full when planned is
                # live: its count is read on the device (such nodes are planned
                # up to their capacity); `valid` is the count at planning time
                n_len, n_cap, n_kids = int(nodes[node][3]), int(nodes[node][4]), int(kids[node])
                assert tin * 32 < (n_cap if live_mode and n_kids == 0 else n_len)
                assert 0 <= valid <= max(0, min(32, n_len - 32 * tin))
                if v < 0:
                    assert live_mode and n_kids == 0 and valid < 32
                    assert -1 - v < n_l and -1 - v not in used_live
                    used_live.add(-1 - v)
                    assert tuple(live[-1 - v]) == (node, 32 * tin)
                else:
                    assert v == valid == min(32, n_len - 32 * tin) and 1 <= v <= 32
                    assert valid == 32 or not live_mode or n_kids > 0 or n_len == n_cap
            for j in range(nl):
                x = int(rowsets[rb + j])
                assert 0 <= x < len(leaves) and sg[seg + j] == (x * hq + g * G) * d
                e = entry.get((x, g), 0)
                entry[(x, g)] = e + 1
                assert dst[seg + j] == (base[(x, g)] + e) * G
        assert used_live == set(range(n_l))
    assert entry == count


def _stream_costs(pieces, n_streams, q_cost=1.2, cut_q=False):
    """The planner's estimated cost per stream: KV tiles by piece height,
    plus the query tiles of each sequence's first piece (and with cut_q also
    those that a piece continuing a sequence cut at a stream boundary loads
    again, which the planner leaves out as a per-stream overhead)."""
    cost = np.zeros(n_streams)
    prev = None
    for pc in pieces:
        key = (pc[8], pc[0], pc[3])  # run, rowset, KV head
        first = key != prev
        prev = key
        cost[pc[9]] += pc[5] * _tile_cost(pc[2]) + (q_cost * pc[11] if first or cut_q else 0.0)
    return cost


@pytest.mark.parametrize("cfg,bt", [(1, 64), (2, 64), (4, 64), (6, 64), (1, 16), (4, 16), (2, 32)])
def test_plan_covers_each_chain_token_once(cfg, bt):
    log = build_call_log(cfg)
    from workloads import CONFIGS
    c = CONFIGS[cfg]
    ctx = host_ctx(hq=c.hq, hkv=c.hkv, d=c.d, block_tokens=bt)
    replay_host(ctx, log)
    model = oracle_model(log, block_tokens=bt)
    p_t, tiles_t, _ = _plan_checks(ctx, model, log.leaves, 0)
    p_n, tiles_n, _ = _plan_checks(ctx, model, log.leaves, 1)
    # the tree plan streams every node once per leaf group; the naive plan once per leaf
    tree_tok = sum(int(t[3]) for pc in p_t for t in tiles_t[pc[10]:pc[10] + pc[5]])
    naive_tok = sum(int(t[3]) for pc in p_n for t in tiles_n[pc[10]:pc[10] + pc[5]])
    logical = sum(model.chain_len(x) for x in log.leaves) * c.hkv
    assert naive_tok == logical
    assert tree_tok <= naive_tok


@pytest.mark.parametrize("cfg,cus,xcds,regime", [
    (2, 256, 8, "one round"), (4, 256, 8, "guided"),
    # other machine shapes: a 304-CU part (one round, 608 streams) and a
    # single 32-CU die (config 2 then takes several rounds)
    (2, 304, 8, "one round"), (2, 32, 1, "guided"), (4, 80, 4, "guided"),
])
def test_stream_sizes(cfg, cus, xcds, regime):
    """One round of resident workgroups (at most 2 CUs x 192 cost units): one
    stream per slot, estimated cost in proportion to the speed of its slot and
    XCD to within about two tiles.  More work: guided sizes, each stream 1/2
    of an even (2 CUs)-way share of the work not yet assigned scaled by its
    XCD's speed (relative to the mean), clamped to [8, 192]."""
    log = build_call_log(cfg)
    from workloads import CONFIGS
    c = CONFIGS[cfg]
    ctx = host_ctx(hq=c.hq, hkv=c.hkv, d=c.d)
    if (cus, xcds) != (256, 8):
        ctx.set_device_shape(cus, xcds)
    replay_host(ctx, log)
    model = oracle_model(log)
    slots = 2 * cus
    seen = set()
    for mode in (0, 1):
        pieces, tiles, n_streams = _plan_checks(ctx, model, log.leaves, mode)
        cost = _stream_costs(pieces, n_streams)
        total = cost.sum()
        if total <= slots * 192:
            seen.add("one round")
            assert n_streams == min(len(tiles), slots) or n_streams >= 0.95 * min(len(tiles), slots)
            rel = cost / _speed(np.arange(n_streams), cus, xcds)
            assert rel.max() <= rel.mean() + 2 * 2.6 + 2.0, (mode, rel.mean(), rel.max())
            # (the last stream takes the remainder, which may be short)
            assert rel[:-1].min() >= rel.mean() - 2 * 2.6 - 2.0 or n_streams < slots
        else:
            seen.add("guided")
            kv = _stream_costs(pieces, n_streams, q_cost=0.0)
            before = np.concatenate([[0.0], np.cumsum(kv)[:-1]])
            die = np.where((np.arange(n_streams) % xcds) % 2 == 1, ODD_XCD_SPEED, 1.0) if xcds > 1 \
                else np.ones(n_streams)
            xs = die / (np.mean(die[:xcds]) if xcds > 1 else 1.0)
            want = np.clip(xs * (kv.sum() - before) / (2 * slots), 8, 192)
            # a stream closes on the first tile that reaches its size (plus the
            # query tiles of a piece it opens), or finishes the sequence it is
            # in when at most its size (kSnapFinish = 1) is left of it
            assert (cost[:-1] <= 2.0 * want[:-1] + 2 * 2.6 + 2.5).all()
            # it closes early only at a sequence boundary within half its size
            # (kSnapEarly = 0.5), or when one of its tables (tiles, query
            # segments, pieces) fills
            hdr = ctx.export_blocks(log.leaves, mode)[:, :3]
            table_full = (hdr[:, 1] >= 256 - 3) | (hdr[:, 2] > 256 - 128 // (c.hq // c.hkv)) | (hdr[:, 0] >= 127)
            short = cost[:-1] < 0.5 * want[:-1] - 2 * 2.6 - 2.5
            assert table_full[:-1][short].all()
            assert cost[-1] <= 2.0 * want[-1] + 2 * 2.6 + 2.5
    assert regime in seen


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


def test_live_plans_outlive_appends():
    """With device lengths, a plan covers every unfrozen node up to its
    capacity (tiles not yet full are live) and is reused across appends --
    also ones that cross tile and block boundaries -- until the next fork."""
    log = build_call_log(1)
    from workloads import CONFIGS
    c = CONFIGS[1]
    ctx = host_ctx(hq=c.hq, hkv=c.hkv, d=c.d, live=True)
    replay_host(ctx, log)
    model = oracle_model(log)
    # a new 100-token segment under every leaf (the next step of Alg. 1), 5 tokens in
    leaves = []
    for x in log.leaves:
        kid, = ctx.fork(x, 1, 100)
        assert model.fork(x, 1, 100) == [kid]
        leaves.append(kid)
    ctx.kv_commit(leaves, [5] * len(leaves))
    model.append(leaves, [5] * len(leaves))
    for mode in (0, 1):
        _plan_checks(ctx, model, leaves, mode)
    b0 = ctx.export_blocks(leaves, 0)
    assert b0[:, 3].sum() == len(leaves) * c.hkv * 4      # 100 tokens: 4 tiles per leaf and KV head, none full
    for step in (1, 40, 53):                            # 6, 46 (past 32), 99 (past 64)
        ctx.kv_commit(leaves, [step] * len(leaves))
        model.append(leaves, [step] * len(leaves))
        _plan_checks(ctx, model, leaves, 0)
        assert np.array_equal(ctx.export_blocks(leaves, 0), b0)   # the same plan serves every step
    # a fork changes the shape: a new plan; the frozen node is static, the others
    # have one live tile left (tokens 96..99 of 100)
    ctx.fork(leaves[0], 2, 64)
    model.fork(leaves[0], 2, 64)
    b1 = ctx.export_blocks(leaves, 0)
    assert not np.array_equal(b1, b0) and b1[:, 3].sum() == (len(leaves) - 1) * c.hkv
    _plan_checks(ctx, model, leaves, 0)


def test_static_plans_follow_appends():
    """Without device lengths every append re-plans (counts baked in)."""
    log = build_call_log(1)
    from workloads import CONFIGS
    c = CONFIGS[1]
    ctx = host_ctx(hq=c.hq, hkv=c.hkv, d=c.d)
    replay_host(ctx, log)
    leaves = list(log.leaves)
    b0 = ctx.export_blocks(leaves, 0)
    assert (b0[:, 3] == 0).all()
    nodes = ctx.export_nodes()
    frozen = set(int(p) for p in nodes[:, 0] if p >= 0)
    grow = [x for x in leaves if nodes[x][3] < nodes[x][4] and x not in frozen]
    if grow:
        ctx.kv_commit(grow[:1], [1])
        assert not np.array_equal(ctx.export_blocks(leaves, 0), b0)


def test_misaligned_fallback_workload_shape():
    """The fork-variant workload cuts 1024-token segments at their 512-token
    midpoint (the misaligned fallback) and re-forks interior nodes; every
    node starts on a 512-token boundary after the 512-token prompt."""
    log = build_call_log(6)
    cuts = [op for op in log.ops if op[0] == "fork_at"]
    assert len(cuts) >= 10 and all(op[2] == 512 for op in cuts)
    model = oracle_model(log)
    starts = {nd["start"] for nd in model.nodes if nd["parent"] >= 0}
    assert all((s - 512) % 512 == 0 for s in starts) and any((s - 512) % 1024 for s in starts)
    kids = {}
    for i, nd in enumerate(model.nodes):
        kids.setdefault(nd["parent"], []).append(i)
    assert any(len(v) > 2 for k, v in kids.items() if k >= 0)      # re-forks of a node that had children
    per_tree = {}
    for x in log.leaves:
        per_tree[model.nodes[x]["tree_id"]] = per_tree.get(model.nodes[x]["tree_id"], 0) + 1
    assert max(per_tree.values()) == 16
