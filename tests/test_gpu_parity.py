"""GPU parity: the HIP path (through the C-ABI) vs the fp64 oracle.

Bar: max |out - oracle| <= 2e-3 and max |lse - oracle| <= 2e-3 over every
compared element (bf16 inputs, fp32 accumulation).  Every workload is
compared in full, at full size: every leaf of every tree (the oracle works
one tree at a time).  Both the cascade (tree) path and the per-leaf
baseline are checked, plus determinism and edge cases (ragged tails,
zero-length nodes, one-token chains, duplicate and interior leaves, GQA
group sizes from 1 to 48, D = 64 and 128).
"""

from __future__ import annotations

import numpy as np
import pytest

from oracle import attention as A
from oracle import metadata as M
from tests.oracle_pins import _Log, random_tiny_tree
from workloads import CONFIGS, Config, build_call_log, query_bits

TOL = 2e-3

pytestmark = pytest.mark.gpu


def _oracle(dt, positions=None):
    log, cfg = dt.log, dt.cfg
    model = M.replay(log, cfg.block_tokens, dt.num_blocks, max(log.n_nodes, 1))
    q = query_bits(cfg.seed, 0, len(log.leaves), cfg.hq, cfg.d)
    return A.tree_decode(model, dt.data, log.leaves, q, cfg.scale, positions=positions)


def _check(dt, mode, positions=None, tag=""):
    import torch
    out, lse = dt.decode(mode)
    torch.cuda.synchronize()
    ref, ref_lse = _oracle(dt, positions)
    o = out.cpu().numpy()
    l = lse.cpu().numpy()
    if positions is not None:
        o, l = o[positions], l[positions]
    err = float(np.abs(o - ref).max())
    err_l = float(np.abs(l - ref_lse).max())
    print(f"[parity {tag} mode={mode}] max|out-oracle|={err:.3e} mean={float(np.abs(o - ref).mean()):.3e} "
          f"max|lse-oracle|={err_l:.3e}", flush=True)
    assert np.isfinite(o).all()
    assert err <= TOL and err_l <= TOL
    return out


def _dt(cfg_id=None, cfg=None, log=None, **kw):
    from workloads.device import DeviceTree
    print(f"[build cfg={cfg_id or (cfg and cfg.name)}]", flush=True)
    return DeviceTree(cfg_id=cfg_id, cfg=cfg, log=log, keep_host_data=True, **kw)


@pytest.mark.parametrize("cfg_id", [1, 2])
def test_small_configs_full(cfg_id):
    dt = _dt(cfg_id)
    for mode in (0, 1):
        _check(dt, mode, tag=f"cfg{cfg_id}")


def test_determinism_and_identical_paths():
    import torch
    dt = _dt(2)
    a, _ = dt.decode(0)
    b, _ = dt.decode(0)
    torch.cuda.synchronize()
    assert torch.equal(a, b)
    # duplicated leaves with the same query give bitwise identical rows
    leaves = dt.leaves[:3] + dt.leaves[:3]
    q = torch.cat([dt.q[:3], dt.q[:3]])
    out = torch.empty((6, dt.cfg.hq, dt.cfg.d), dtype=torch.float32, device="cuda")
    ws = torch.empty(dt.ctx.workspace_size(leaves, 0), dtype=torch.uint8, device="cuda")
    dt.ctx.tree_decode(leaves, q, dt.cfg.scale, out, None, ws)
    torch.cuda.synchronize()
    assert torch.equal(out[:3], out[3:])


def _random_cfg(seed, hq, hkv, d):
    return Config(f"random-{seed}", 1000 + seed, hq, hkv, d, gen=None)


@pytest.mark.parametrize("seed,hq,hkv,d", [
    (1, 4, 1, 64), (2, 7, 1, 128), (3, 8, 8, 128), (4, 6, 3, 64), (5, 28, 4, 128),
    (6, 40, 8, 128), (7, 16, 2, 64), (8, 5, 1, 128), (9, 3, 3, 64), (10, 2, 1, 128),
    (11, 32, 2, 128), (12, 48, 1, 64), (13, 14, 1, 128), (14, 12, 1, 64),
])
def test_random_trees(seed, hq, hkv, d):
    ops, leaves, rows, _ = random_tiny_tree(seed, max_leaves=10, max_tokens=400)
    log = _Log(ops, leaves or [0], rows)
    log.n_nodes = len(rows)
    cfg = _random_cfg(seed, hq, hkv, d)
    dt = _dt(cfg=cfg, log=log)
    for mode in (0, 1):
        _check(dt, mode, tag=f"rand{seed}")


@pytest.mark.parametrize("bt", [64, 16])
def test_ragged_and_degenerate_shapes(bt):
    """One-token chains, a leaf whose own node is empty, tails of 1 and 63
    tokens, a chain crossing many partial tiles, an interior node decoded as a
    leaf, and a 64-token-aligned chain; pools in 64- and 16-token blocks."""
    import dataclasses
    ops = [("root", 1), ("append", [0], [1]),                   # 0: one token
           ("root", 200), ("append", [1], [129]),               # 1: 2 full tiles + 1
           ("fork", 1, 3, 64), ("append", [2, 3, 4], [63, 0, 64]),
           ("fork", 2, 2, 5), ("append", [5, 6], [1, 5]),
           ("root", 64), ("append", [7], [64])]
    rows = {0: 1, 1: 129, 2: 63, 3: 0, 4: 64, 5: 1, 6: 5, 7: 64}
    leaves = [0, 3, 5, 6, 2, 1, 7, 4, 0]
    log = _Log(ops, leaves, rows)
    log.n_nodes = 8
    for (hq, hkv, d) in ((28, 4, 128), (4, 1, 64)):
        dt = _dt(cfg=dataclasses.replace(_random_cfg(77, hq, hkv, d), block_tokens=bt), log=log)
        for mode in (0, 1):
            _check(dt, mode, tag=f"ragged-d{d}-B{bt}")


@pytest.mark.parametrize("bt", [16, 32])
def test_block_sizes(bt):
    """Pools reserved in 16- and 32-token blocks.  With B = 16 a node starts
    on any 16-row boundary, so its 32-token tiles straddle the pool's 32-row
    lines and a node's last tile reaches into the next node's rows.  The tiny
    workload (16-token segments, one block each at B = 16), the single
    7,680-token tree and random trees, in both modes."""
    import dataclasses
    for cfg_id in (1, 2):
        cfg = dataclasses.replace(CONFIGS[cfg_id], block_tokens=bt)
        dt = _dt(cfg=cfg, log=build_call_log(cfg_id))
        for mode in (0, 1):
            _check(dt, mode, tag=f"cfg{cfg_id}-B{bt}")
    for seed, hq, hkv, d in ((3, 8, 8, 128), (4, 6, 3, 64), (5, 28, 4, 128)):
        ops, leaves, rows, _ = random_tiny_tree(seed, max_leaves=10, max_tokens=400)
        log = _Log(ops, leaves or [0], rows)
        log.n_nodes = len(rows)
        dt = _dt(cfg=dataclasses.replace(_random_cfg(seed, hq, hkv, d), block_tokens=bt), log=log)
        for mode in (0, 1):
            _check(dt, mode, tag=f"rand{seed}-B{bt}")


def _oracle_by_tree(dt):
    """The oracle over every call position, one tree at a time (the oracle's
    per-node cache then holds one tree's fp64 K/V at a time)."""
    log, cfg = dt.log, dt.cfg
    model = M.replay(log, cfg.block_tokens, dt.num_blocks, max(log.n_nodes, 1))
    q = query_bits(cfg.seed, 0, len(log.leaves), cfg.hq, cfg.d)
    by_tree = {}
    for p, x in enumerate(log.leaves):
        by_tree.setdefault(model.nodes[x]["tree_id"], []).append(p)
    ref = np.empty((len(log.leaves), cfg.hq, cfg.d))
    ref_lse = np.empty((len(log.leaves), cfg.hq))
    for t, pos in sorted(by_tree.items()):
        o, l = A.tree_decode(model, dt.data, log.leaves, q, cfg.scale, positions=pos)
        ref[pos], ref_lse[pos] = o, l
    return ref, ref_lse


@pytest.mark.parametrize("cfg_id", [3, 4, 5, 6])
def test_large_configs_every_leaf(cfg_id):
    """The full-size workloads, every leaf of every tree against the oracle,
    in both modes; the two modes (different plans: stream cuts, partial slots)
    also agree with each other."""
    import torch
    dt = _dt(cfg_id)
    outs = {}
    for mode in (0, 1):
        out, lse = dt.decode(mode)
        torch.cuda.synchronize()
        outs[mode] = (out.cpu().numpy(), lse.cpu().numpy())
        assert np.isfinite(outs[mode][0]).all() and np.isfinite(outs[mode][1]).all()
    print(f"[cfg{cfg_id}] {len(dt.leaves)} leaves decoded; oracle ...", flush=True)
    ref, ref_lse = _oracle_by_tree(dt)
    for mode in (0, 1):
        o, l = outs[mode]
        err, err_l = float(np.abs(o - ref).max()), float(np.abs(l - ref_lse).max())
        print(f"[parity cfg{cfg_id} all {len(dt.leaves)} leaves mode={mode}] max|out-oracle|={err:.3e} "
              f"mean={float(np.abs(o - ref).mean()):.3e} max|lse-oracle|={err_l:.3e}", flush=True)
        assert err <= TOL and err_l <= TOL
    assert float(np.abs(outs[0][0] - outs[1][0]).max()) <= TOL
    del dt
    torch.cuda.empty_cache()


@pytest.mark.parametrize("cfg_id,hq,hkv", [(2, 16, 2), (4, 32, 4)])
def test_head_dim_64_full_size(cfg_id, hq, hkv):
    """D = 64 at full size: the 16-leaf 7,680-token tree (one round of streams)
    and the irregular 32-prompt trees (several rounds; 32-leaf roots give 256
    rows at G = 8, cut into two leaf groups), every leaf against the oracle
    in both modes."""
    import dataclasses
    import torch
    cfg = dataclasses.replace(CONFIGS[cfg_id], hq=hq, hkv=hkv, d=64)
    dt = _dt(cfg=cfg, log=build_call_log(cfg_id))
    outs = {}
    for mode in (0, 1):
        out, lse = dt.decode(mode)
        torch.cuda.synchronize()
        outs[mode] = (out.cpu().numpy(), lse.cpu().numpy())
        assert np.isfinite(outs[mode][0]).all() and np.isfinite(outs[mode][1]).all()
    ref, ref_lse = _oracle_by_tree(dt)
    for mode in (0, 1):
        o, l = outs[mode]
        err, err_l = float(np.abs(o - ref).max()), float(np.abs(l - ref_lse).max())
        print(f"[parity cfg{cfg_id} D=64 all {len(dt.leaves)} leaves mode={mode}] max|out-oracle|={err:.3e} "
              f"max|lse-oracle|={err_l:.3e}", flush=True)
        assert err <= TOL and err_l <= TOL
    del dt
    torch.cuda.empty_cache()


@pytest.mark.parametrize("n_leaves,hq,hkv", [(1024, 28, 4), (4096, 8, 8)])
def test_wide_root(n_leaves, hq, hkv):
    """One 1,000-token root under 1,024 or 4,096 one- to three-token leaves:
    the root's rows (leaves x G) are cut into dozens of leaf groups of at most
    128 rows, streams hold many pieces and up to a full table of query
    segments, and every leaf's key merges the root's partial with its own."""
    import torch
    rng = np.random.default_rng(n_leaves)
    own = [int(x) for x in rng.integers(1, 4, n_leaves)]
    ops = [("root", 1000), ("append", [0], [1000]), ("fork", 0, n_leaves, 64),
           ("append", list(range(1, n_leaves + 1)), own)]
    rows = {0: 1000, **{1 + i: own[i] for i in range(n_leaves)}}
    log = _Log(ops, list(range(1, n_leaves + 1)), rows)
    log.n_nodes = n_leaves + 1
    dt = _dt(cfg=_random_cfg(200 + hq, hq, hkv, 128), log=log)
    pieces, _, _, ns = dt.ctx.export_plan(dt.leaves, 0)
    print(f"[wide root] {n_leaves} leaves: {ns} streams, {len(pieces)} pieces, "
          f"{len({int(p[0]) for p in pieces if p[1] > 1})} root leaf groups", flush=True)
    for mode in (0, 1):
        _check(dt, mode, tag=f"wide-root-{n_leaves}")
    del dt
    torch.cuda.empty_cache()


def test_many_entries_per_key():
    """Leaves whose (leaf, KV head) keys collect hundreds of partial entries
    (a 40,000-token root cut over every stream, then a short fork): the
    combine's rounds past the first 64 entries."""
    import torch
    ops = [("root", 40_000), ("append", [0], [40_000]), ("fork", 0, 2, 64), ("append", [1, 2], [17, 64])]
    log = _Log(ops, [1, 2, 0], {0: 40_000, 1: 17, 2: 64})
    log.n_nodes = 3
    dt = _dt(cfg=_random_cfg(91, 8, 2, 128), log=log)
    pieces, rowsets, _, _ = dt.ctx.export_plan(dt.leaves, 0)
    count = {}
    for pc in pieces:
        for x in rowsets[pc[0]:pc[0] + pc[1]]:
            count[(int(x), int(pc[3]))] = count.get((int(x), int(pc[3])), 0) + 1
    print(f"[entries per key] {sorted(count.values())}", flush=True)
    assert min(count.values()) > 128
    for mode in (0, 1):
        _check(dt, mode, tag="many-entries")
    del dt
    torch.cuda.empty_cache()


def test_compact_plan_many_entries_per_key():
    """A plan with compact partial slots (block floating-point rows) whose keys
    hold 59-74 entries each: a 60,000-token root under 8 leaves, G = 8, 8 KV
    heads, cut over every stream -- the compact combine's later rows and its
    second batch of 64 entries."""
    import torch
    n = 8
    ops = [("root", 60_000), ("append", [0], [60_000]), ("fork", 0, n, 64),
           ("append", list(range(1, n + 1)), [5] * n)]
    log = _Log(ops, list(range(1, n + 1)), {0: 60_000, **{1 + i: 5 for i in range(n)}})
    log.n_nodes = n + 1
    dt = _dt(cfg=_random_cfg(93, 64, 8, 128), log=log)
    pieces, rowsets, _, _ = dt.ctx.export_plan(dt.leaves, 0)
    count = {}
    for pc in pieces:
        for x in rowsets[pc[0]:pc[0] + pc[1]]:
            count[(int(x), int(pc[3]))] = count.get((int(x), int(pc[3])), 0) + 1
    rows = sum(count.values()) * 8
    print(f"[entries per key] {min(count.values())}-{max(count.values())}; workspace "
          f"{dt.ctx.workspace_size(dt.leaves, 0)} B for {rows} partial rows", flush=True)
    assert max(count.values()) > 64
    # compact slots: rows of D / 2 dwords plus (m, l), not fp32 rows at a stride of the largest count
    assert dt.ctx.workspace_size(dt.leaves, 0) < rows * (128 * 4 + 8)
    for mode in (0, 1):
        _check(dt, mode, tag="compact-many-entries")
    del dt
    torch.cuda.empty_cache()


def test_shared_workspace_between_contexts():
    """One workspace buffer used in turn by two contexts (different shapes and
    plans) and filled with 0xFF before every call: the plans live in memory
    each context owns and every partial the combine reads is written by the
    same call, so each context keeps giving its own, bitwise equal results."""
    import torch
    t1, t2 = _dt(1), _dt(2)
    refs = {}
    for t in (t1, t2):
        for mode in (0, 1):
            out, _ = t.decode(mode)
            refs[(id(t), mode)] = out.clone()
    torch.cuda.synchronize()
    nbytes = max(t.ctx.workspace_size(t.leaves, m) for t in (t1, t2) for m in (0, 1))
    ws = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    for it in range(2):
        for t in (t1, t2):
            for mode in (0, 1):
                ws.fill_(255)
                out, _ = t.decode(mode, ws=ws)
                torch.cuda.synchronize()
                print(f"[shared workspace it={it} cfg={t.cfg.name} mode={mode}]", flush=True)
                assert torch.equal(out, refs[(id(t), mode)])


def _poisoned_kv(monkeypatch, node, tok, g, d, bits):
    """Makes the workload generators give V[node][tok, g, d] the bf16 pattern
    `bits` (a NaN or an infinity)."""
    import workloads.device as wd
    gen1, genm = wd.node_kv_bits, wd.many_node_kv_bits

    def poison(o, kv):
        if o != node:
            return kv
        k, v = kv
        v = v.copy()
        v[tok, g, d] = bits
        return k, v

    monkeypatch.setattr(wd, "node_kv_bits", lambda seed, o, rows, hkv, dd: poison(o, gen1(seed, o, rows, hkv, dd)))
    monkeypatch.setattr(wd, "many_node_kv_bits",
                        lambda seed, nr, hkv, dd, threads=None: [poison(o, kv) for (o, _), kv in
                                                                 zip(nr, genm(seed, nr, hkv, dd, threads))])


def _four_level_tree(fan, tokens):
    """A root and three levels of `fan`-way forks; node ids in fork order."""
    ops = [("root", tokens[0]), ("append", [0], [tokens[0]])]
    rows = {0: tokens[0]}
    level, nxt = [0], 1
    for depth in range(1, 4):
        new = []
        for p in level:
            ops.append(("fork", p, fan, tokens[depth]))
            kids = list(range(nxt, nxt + fan))
            nxt += fan
            ops.append(("append", kids, [tokens[depth]] * fan))
            rows.update({c: tokens[depth] for c in kids})
            new += kids
        level = new
    log = _Log(ops, level, rows)
    log.n_nodes = nxt
    return log


@pytest.mark.parametrize("kind", ["nan", "inf"])
@pytest.mark.parametrize("shape", ["strided", "compact"])
def test_non_finite_values_stay_non_finite(kind, shape, monkeypatch):
    """One V entry of the shared root set to NaN or +inf: the outputs of that
    column (every leaf, the KV head's query heads) are non-finite, as in the
    oracle, and every other output matches it.  In a plan with compact
    partial slots the non-finite value spoils its whole 4-value d-group of
    the partial rows (the block format keeps no finite values beside a
    non-finite one), so there the outputs of that d-group's columns are
    non-finite too -- never a finite stand-in."""
    import torch
    g, d = 1, 37
    _poisoned_kv(monkeypatch, 0, 123, g, d, 0x7FC0 if kind == "nan" else 0x7F80)
    if shape == "strided":
        log = _four_level_tree(2, [300, 70, 50, 30])
        cfg = _random_cfg(95, 8, 2, 128)
    else:
        log = _four_level_tree(4, [2048, 512, 256, 64])
        cfg = _random_cfg(96, 64, 8, 128)
    dt = _dt(cfg=cfg, log=log)
    G = cfg.hq // cfg.hkv
    pieces, rowsets, _, _ = dt.ctx.export_plan(dt.leaves, 0)
    count = {}
    for pc in pieces:
        for x in rowsets[pc[0]:pc[0] + pc[1]]:
            count[(int(x), int(pc[3]))] = count.get((int(x), int(pc[3])), 0) + 1
    ws = dt.ctx.workspace_size(dt.leaves, 0)
    # strided slots hold fp32 rows for the largest entry count of every key
    compact = ws < len(count) * max(count.values()) * G * (cfg.d * 4 + 8)
    print(f"[non-finite {kind} {shape}] leaves {len(dt.leaves)} workspace {ws} B compact={compact}", flush=True)
    assert compact == (shape == "compact")
    ref, ref_lse = _oracle(dt)
    bad_ref = ~np.isfinite(ref)
    assert bad_ref[:, g * G:(g + 1) * G, d].all() and bad_ref.sum() == len(dt.leaves) * G
    group = np.zeros_like(bad_ref)
    group[:, g * G:(g + 1) * G, 4 * (d // 4):4 * (d // 4) + 4] = True
    for mode in (0, 1):
        out, lse = dt.decode(mode)
        torch.cuda.synchronize()
        o, l = out.cpu().numpy(), lse.cpu().numpy()
        bad = ~np.isfinite(o)
        print(f"[non-finite {kind} {shape} mode={mode}] non-finite outputs {int(bad.sum())} "
              f"(oracle {int(bad_ref.sum())})", flush=True)
        assert (bad | ~bad_ref).all(), "a non-finite oracle output came out finite"
        assert not (bad & ~group).any(), "non-finite outputs outside the poisoned d-group"
        ok = ~bad & ~bad_ref
        assert float(np.abs(o[ok] - ref[ok]).max()) <= TOL
        assert np.isfinite(l).all() and float(np.abs(l - ref_lse).max()) <= TOL
    del dt
    torch.cuda.empty_cache()
