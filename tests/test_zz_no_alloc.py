"""The decode entry point that allocates nothing, through the C-ABI.

``treepo_tree_decode_noalloc`` runs the cascade decode with its plan image and
partial slots in the library's static device scratch.  Its output is checked
against ``treepo_tree_decode`` (workspace from the caller) on the same inputs
to the parity bar (|diff| <= 2e-3; both run the same plan through the same
kernels, so the results are in fact bitwise equal), over calls in a row:
the full config-2 tree, then a smaller decode of another context (the scratch
then holds another plan), then config 2 again (its plan uploaded again), and
a context with device-resident lengths across an append.
"""

from __future__ import annotations

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

TOL = 2e-3


def _same(a, b):
    import torch
    assert torch.isfinite(a).all()
    assert float((a - b).abs().max()) <= TOL
    assert torch.equal(a, b)


def _pair(dt, leaves, q):
    """(workspace decode, no-alloc decode) outputs for these leaves; the
    no-alloc call goes first, so it is the one that uploads a stale length
    table."""
    import torch
    c = dt.cfg
    n = len(leaves)
    out = torch.full((n, c.hq, c.d), float("nan"), dtype=torch.float32, device="cuda")
    lse = torch.full((n, c.hq), float("nan"), dtype=torch.float32, device="cuda")
    dt.ctx.tree_decode_noalloc(leaves, q, c.scale, out, lse)
    ref = torch.empty_like(out)
    ref_lse = torch.empty_like(lse)
    ws = torch.empty(max(dt.ctx.workspace_size(leaves, 0), 256), dtype=torch.uint8, device="cuda")
    dt.ctx.tree_decode(leaves, q, c.scale, ref, ref_lse, ws)
    torch.cuda.synchronize()
    return ref, ref_lse, out, lse


def test_noalloc_decode_matches_workspace_decode():
    import torch
    from workloads.device import DeviceTree
    print("[no-alloc] build config 2 and config 1", flush=True)
    big = DeviceTree(cfg_id=2)
    small = DeviceTree(cfg_id=1)
    # 1: the whole config-2 tree
    ref, ref_lse, out, lse = _pair(big, big.leaves, big.q)
    _same(out, ref)
    _same(lse, ref_lse)
    print("[no-alloc] config 2 equal", flush=True)
    # 2: a smaller input on another context (another plan in the scratch)
    sub = small.leaves[:5]
    q = small.q[:5].contiguous()
    ref, ref_lse, out, lse = _pair(small, sub, q)
    _same(out, ref)
    _same(lse, ref_lse)
    print("[no-alloc] config 1, 5 leaves equal", flush=True)
    # 3: config 2 again: its plan is uploaded into the scratch again
    ref, ref_lse, out, lse = _pair(big, big.leaves, big.q)
    _same(out, ref)
    _same(lse, ref_lse)
    print("[no-alloc] config 2 again equal", flush=True)
    del big, small
    torch.cuda.empty_cache()


def test_noalloc_decode_with_device_lengths():
    """Device-resident lengths: the length table goes up from pageable
    memory, and after each append the same plan serves the next step."""
    import torch
    from workloads import CONFIGS, CallLog, build_call_log
    from workloads.device import DeviceTree
    base = build_call_log(1)
    ops, rows, nid, kids = list(base.ops), dict(base.rows), base.n_nodes, []
    for x in base.leaves:          # an empty 8-token segment under every leaf
        ops.append(("fork", x, 1, 8))
        rows[nid] = 0
        kids.append(nid)
        nid += 1
    dt = DeviceTree(cfg=CONFIGS[1], log=CallLog(ops=ops, step_append=None, leaves=kids, rows=rows, n_nodes=nid),
                    live=True)
    n = len(kids)
    g = torch.Generator(device="cuda").manual_seed(3)
    kv = [torch.randn(n, dt.cfg.hkv, dt.cfg.d, device="cuda", generator=g).to(torch.bfloat16) for _ in range(2)]
    for step in range(3):
        ref, ref_lse, out, lse = _pair(dt, kids, dt.q)
        _same(out, ref)
        _same(lse, ref_lse)
        print(f"[no-alloc] device lengths, step {step} equal", flush=True)
        dt.ctx.kv_append(kids, [1] * n, kv[step % 2], kv[1 - step % 2])
    assert np.isfinite(out.cpu().numpy()).all()
