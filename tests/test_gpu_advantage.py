"""GPU parity: the TreePO advantage kernel (through the C-ABI) vs the fp64 oracle.

Bar: max |adv - oracle| <= 1e-6 (fp64 arithmetic on the device, fp32 output).
Leaf sets of the five workloads with 0/1 and N(0,1) rewards, both
aggregations; edge cases: rejected queries (all rewards equal), duplicate and
interior leaves, a root decoded as a trajectory, one query with all rewards
equal (every advantage 0); determinism.
"""

from __future__ import annotations

import numpy as np
import pytest

from oracle import advantage as ADV
from tests.lib_helpers import host_ctx, oracle_model, replay_host
from tests.advantage_pins import random_forest
from workloads import CONFIGS, build_call_log

TOL = 1e-6

pytestmark = pytest.mark.gpu


def _gpu_adv(ctx, leaves, R, weighting):
    import torch
    rw = torch.tensor(np.asarray(R, dtype=np.float32), device="cuda")
    out = torch.full((len(leaves),), float("nan"), dtype=torch.float32, device="cuda")
    ws = torch.empty(max(ctx.advantage_workspace_size(leaves), 256), dtype=torch.uint8, device="cuda")
    ctx.tree_advantage(leaves, rw, out, ws, weighting)
    torch.cuda.synchronize()
    return out.cpu().numpy().astype(np.float64)


def _check(ctx, parents, leaves, R, tag):
    R32 = np.asarray(R, dtype=np.float32)
    for w, name in ((0, "mean"), (1, "size")):
        got = _gpu_adv(ctx, leaves, R32, w)
        want = ADV.tree_advantage(parents, leaves, R32.astype(np.float64), name)
        err = float(np.abs(got - want).max())
        print(f"[advantage {tag} {name}] n={len(leaves)} max|gpu-oracle|={err:.3e} max|adv|={np.abs(want).max():.3f}",
              flush=True)
        assert np.isfinite(got).all() and err <= TOL


@pytest.mark.parametrize("cfg_id", [1, 2, 3, 4, 5, 6])
def test_configs(cfg_id):
    c = CONFIGS[cfg_id]
    log = build_call_log(cfg_id)
    ctx = host_ctx(hq=c.hq, hkv=c.hkv, d=c.d)
    replay_host(ctx, log)
    parents = [nd["parent"] for nd in oracle_model(log).nodes]
    rng = np.random.default_rng(100 + cfg_id)
    _check(ctx, parents, log.leaves, rng.integers(0, 2, size=len(log.leaves)), f"cfg{cfg_id} 0/1")
    _check(ctx, parents, log.leaves, rng.normal(size=len(log.leaves)), f"cfg{cfg_id} normal")
    if cfg_id in (3, 4):
        # reject every other query: all its trajectories get reward 1
        R = rng.integers(0, 2, size=len(log.leaves)).astype(float)
        roots = [ADV.chain(parents, x)[0] for x in log.leaves]
        order = sorted(set(roots))
        for p, r in enumerate(roots):
            if order.index(r) % 2:
                R[p] = 1.0
        _check(ctx, parents, log.leaves, R, f"cfg{cfg_id} half rejected")


def _build(parents):
    """Creates the forest in the library: roots, then each parent's children
    (consecutive ids) in the order the parents list gives them."""
    ctx = host_ctx()
    ids = {}
    kids = {}
    for x, p in enumerate(parents):
        kids.setdefault(p, []).append(x)
    for x, p in enumerate(parents):
        if x in ids:
            continue
        if p < 0:
            ids[x] = ctx.new_root(64)
        else:
            sib = kids[p]
            got = ctx.fork(ids[p], len(sib), 64)
            for s_, g in zip(sib, got):
                ids[s_] = g
    assert all(ids[x] == x for x in range(len(parents)))
    return ctx


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_random_forests(seed):
    parents, leaves = random_forest(seed, n_roots=4, max_children=3, depth=4)
    ctx = _build(parents)
    rng = np.random.default_rng(seed)
    _check(ctx, parents, leaves, rng.integers(0, 2, size=len(leaves)), f"forest{seed} 0/1")
    _check(ctx, parents, leaves, rng.normal(size=len(leaves)), f"forest{seed} normal")


def test_edge_cases():
    parents, leaves = random_forest(9, n_roots=2, max_children=2, depth=3)
    ctx = _build(parents)
    interior = [x for x in range(len(parents)) if parents[x] >= 0 and x not in leaves][:2]
    lv = leaves + [leaves[0], leaves[3]] + interior + [0]  # duplicates, interior nodes, a root
    rng = np.random.default_rng(9)
    _check(ctx, parents, lv, rng.integers(0, 2, size=len(lv)), "duplicates+interior+root")
    # one query, all rewards equal: every advantage 0
    got = _gpu_adv(ctx, leaves, np.ones(len(leaves), dtype=np.float32), 0)
    assert np.all(got == 0.0)


def test_deterministic():
    c = CONFIGS[3]
    log = build_call_log(3)
    ctx = host_ctx(hq=c.hq, hkv=c.hkv, d=c.d)
    replay_host(ctx, log)
    R = np.random.default_rng(5).normal(size=len(log.leaves)).astype(np.float32)
    a = _gpu_adv(ctx, log.leaves, R, 0)
    b = _gpu_adv(ctx, log.leaves, R, 0)
    assert np.array_equal(a, b)
