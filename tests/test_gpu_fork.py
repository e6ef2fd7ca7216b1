"""GPU parity after fallbacks inside a segment (treepo_fork_at).

A split leaves the pool untouched: the tail node reads the blocks the node
held, so every existing trajectory must decode to the same result as before
the split, and the new branches (filled after the split) must decode like the
oracle.  Bar: max |out - oracle| <= 2e-3 and max |lse - oracle| <= 2e-3, both
for the cascade path and the per-leaf baseline, with static and live
(device-resident) node lengths.
"""

from __future__ import annotations

import numpy as np
import pytest

from oracle import attention as A
from oracle import metadata as M
from tests.oracle_pins import _Log
from workloads import Config, node_kv_bits, query_bits

TOL = 2e-3
B = 64

pytestmark = pytest.mark.gpu


def _long_tree(seed):
    """Two roots of 150..400 tokens, two levels of 1..3 branches of up to 300
    tokens each (lengths include 0, block multiples and ragged tails)."""
    rng = np.random.default_rng(seed)
    ops, rows, tips, n = [], {}, [], 0
    for _ in range(2):
        ln = int(rng.integers(150, 401))
        ops += [("root", ln), ("append", [n], [ln])]
        rows[n] = ln
        tips.append(n)
        n += 1
    for _ in range(2):
        nxt = []
        for p in tips:
            k = int(rng.integers(1, 4))
            ops.append(("fork", p, k, 300))
            kids = list(range(n, n + k))
            n += k
            lens = [int(rng.choice([0, 64, 128, int(rng.integers(1, 301))])) for _ in kids]
            ops.append(("append", kids, lens))
            rows.update(zip(kids, lens))
            nxt += kids
        tips = nxt
    leaves = [t for t in tips]
    return ops, leaves, rows


class _HostKV:
    """The K/V bit rows every node holds, kept beside the tree on the host."""

    def __init__(self, dt):
        self.rows = {}
        for n, ln in dt.log.rows.items():
            k, v = dt.data(n)
            self.rows[n] = (k[:ln], v[:ln])

    def __call__(self, n):
        return self.rows[n]

    def split(self, x, offset, tail):
        k, v = self.rows[x]
        self.rows[tail] = (k[offset:], v[offset:])
        self.rows[x] = (k[:offset], v[:offset])

    def extend(self, n, k, v):
        k0, v0 = self.rows.get(n, (k[:0], v[:0]))
        self.rows[n] = (np.concatenate([k0, k]), np.concatenate([v0, v]))


def _decode(dt, leaves, q, mode):
    import torch
    c = dt.cfg
    out = torch.empty((len(leaves), c.hq, c.d), dtype=torch.float32, device="cuda")
    lse = torch.empty((len(leaves), c.hq), dtype=torch.float32, device="cuda")
    ws = torch.empty(max(dt.ctx.workspace_size(leaves, mode), 256), dtype=torch.uint8, device="cuda")
    fn = dt.ctx.tree_decode if mode == 0 else dt.ctx.paged_decode_naive
    fn(leaves, q, c.scale, out, lse, ws)
    torch.cuda.synchronize()
    return out.cpu().numpy(), lse.cpu().numpy()


def _check(dt, model, kv, leaves, step, tag):
    c = dt.cfg
    qb = query_bits(c.seed, step, len(leaves), c.hq, c.d)
    q = dt._to_dev(qb)
    ref, ref_lse = A.tree_decode(model, kv, leaves, qb, c.scale)
    res = []
    for mode in (0, 1):
        o, l = _decode(dt, leaves, q, mode)
        err, err_l = float(np.abs(o - ref).max()), float(np.abs(l - ref_lse).max())
        print(f"[fork_at {tag} mode={mode}] leaves={len(leaves)} max|out-oracle|={err:.3e} "
              f"max|lse-oracle|={err_l:.3e}", flush=True)
        assert np.isfinite(o).all()
        assert err <= TOL and err_l <= TOL
        res.append((o, l))
    return res


@pytest.mark.parametrize("seed,hq,hkv,d,live", [
    (1, 8, 1, 128, False), (2, 28, 4, 128, True), (3, 4, 1, 64, False), (4, 16, 2, 64, True),
])
def test_split_then_grow(seed, hq, hkv, d, live):
    from workloads.device import DeviceTree
    ops, leaves, rows = _long_tree(seed)
    log = _Log(ops, leaves, rows)
    log.n_nodes = len(rows) + 64                       # room for tails and new branches
    cfg = Config(f"fork-at-{seed}", 2000 + seed, hq, hkv, d, gen=None)
    print(f"[fork_at build seed={seed} hq={hq} hkv={hkv} d={d} live={live}]", flush=True)
    dt = DeviceTree(cfg=cfg, log=log, keep_host_data=True, extra_blocks=200, live=live)
    model = M.replay(log, B, dt.num_blocks, log.n_nodes)
    kv = _HostKV(dt)
    before = _check(dt, model, kv, leaves, 0, f"s{seed} before")

    # splits at block-aligned offsets inside nodes (interior nodes and leaves, offset 0 included)
    rng = np.random.default_rng(seed + 100)
    traj = {x: x for x in leaves}                      # leaf -> node that now ends its trajectory
    new_kids, n_split = [], 0
    for _ in range(6):
        cand = [i for i, nd in enumerate(model.nodes) if nd["len"] > B]
        x = int(rng.choice(cand))
        offset = B * int(rng.integers(0, (model.nodes[x]["len"] - 1) // B + 1))
        n, cap = int(rng.integers(0, 3)), int(rng.integers(1, 200))
        got = dt.ctx.fork_at(x, offset, n, cap)
        want = model.fork_at(x, offset, n, cap)
        assert got == want
        kids, t = want
        kv.split(x, offset, t)
        for k in kids:
            kv.rows[k] = kv.rows[t][0][:0], kv.rows[t][1][:0]
        for lf, end in traj.items():
            if end == x:
                traj[lf] = t
        new_kids += kids
        n_split += 1
    assert n_split == 6
    exported = dt.ctx.export_nodes()
    assert np.array_equal(exported, np.array([model.record(i) for i in range(len(model.nodes))], np.int32))

    # every old trajectory decodes as before (same query rows)
    ends = [traj[x] for x in leaves]
    after = _check(dt, model, kv, ends, 0, f"s{seed} same trajectories")
    for (o0, l0), (o1, l1) in zip(before, after):
        assert float(np.abs(o0 - o1).max()) <= TOL and float(np.abs(l0 - l1).max()) <= TOL

    # grow the new branches and the tails that are still open leaves
    grow_n, grow_t = [], []
    for i, nd in enumerate(model.nodes):
        if model.n_children[i] == 0 and nd["len"] < nd["cap"] and (i in new_kids or i in ends):
            grow_n.append(i)
            grow_t.append(int(rng.integers(0, nd["cap"] - nd["len"] + 1)))
    ks, vs = [], []
    for n, t in zip(grow_n, grow_t):
        k, v = node_kv_bits(cfg.seed + 1, n, t, hkv, d)
        kv.extend(n, k, v)
        ks.append(k); vs.append(v)
    if grow_n and sum(grow_t):
        dt.ctx.kv_append(grow_n, grow_t, dt._to_dev(np.concatenate(ks)), dt._to_dev(np.concatenate(vs)))
    model.append(grow_n, grow_t)
    final = [e for e in ends] + [k for k in new_kids if model.chain_len(k) > 0]
    final += [x for x in range(len(rows)) if model.n_children[x] > 0 and model.chain_len(x) > 0][:3]
    _check(dt, model, kv, final, 1, f"s{seed} grown")
