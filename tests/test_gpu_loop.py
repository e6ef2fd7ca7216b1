"""GPU parity of segment-level decoding (Sec. 2.2): after a fork, every step
appends one token to each leaf and decodes.  With device lengths
(treepo_config.node_len) one plan serves the whole segment -- tiles fill,
cross 32-token tile and block lines (blocks of 64 and of 16 tokens), and start empty -- and each step
is checked against the fp64 oracle of the tree at that step; without them
every step re-plans.  Same bar as the other parity tests (2e-3).
"""

from __future__ import annotations

import numpy as np
import pytest

from oracle import attention as A
from oracle import metadata as M
from workloads import CONFIGS, CallLog, build_call_log, query_bits

TOL = 2e-3
SEG = 100                      # capacity of the new segment: 3 full tiles and a partial one
CHECK = {1, 2, 31, 32, 33, 63, 64, 65, 99, 100}

pytestmark = pytest.mark.gpu


def _segment_log(cfg_id):
    """The config's tree plus one new SEG-token segment under every leaf."""
    base = build_call_log(cfg_id)
    ops = list(base.ops)
    rows = dict(base.rows)
    nid = base.n_nodes
    leaves = []
    for x in base.leaves:
        ops.append(("fork", x, 1, SEG))
        rows[nid] = SEG          # the generator draws every row the loop will append
        leaves.append(nid)
        nid += 1
    return CallLog(ops=ops, step_append=None, leaves=leaves, rows=rows, n_nodes=nid), base


@pytest.mark.parametrize("live,bt", [(True, 64), (False, 64), (True, 16)])
def test_segment_decode_loop(live, bt):
    import dataclasses
    import torch
    from workloads.device import DeviceTree
    cfg = dataclasses.replace(CONFIGS[1], block_tokens=bt)
    log, base = _segment_log(1)
    print(f"[loop cfg=1 live={live} B={bt}]", flush=True)
    dt = DeviceTree(cfg=cfg, log=log, keep_host_data=True, live=live)
    model = M.replay(log, cfg.block_tokens, dt.num_blocks, log.n_nodes)
    leaves = log.leaves
    q = query_bits(cfg.seed, 0, len(leaves), cfg.hq, cfg.d)
    outs = {m: dt.outputs() for m in (0, 1)}
    wss = {}
    worst = 0.0
    for t in range(1, SEG + 1):
        k, v = dt._stage(leaves, [1] * len(leaves))
        dt.ctx.kv_append(leaves, [1] * len(leaves), k, v)
        for x in leaves:
            dt._len[x] = dt._len.get(x, 0) + 1
        model.append(leaves, [1] * len(leaves))
        if live and t == 1:        # one plan (and workspace) for the whole segment
            wss = {m: dt.workspace(m) for m in (0, 1)}
        for mode in (0, 1):
            out, lse = outs[mode]
            if not live:           # every append re-plans: the workspace size may change
                wss[mode] = dt.workspace(mode)
            fn = dt.ctx.tree_decode if mode == 0 else dt.ctx.paged_decode_naive
            fn(leaves, dt.q, cfg.scale, out, lse, wss[mode])
        if t in CHECK:
            torch.cuda.synchronize()
            ref, ref_lse = A.tree_decode(model, dt.data, leaves, q, cfg.scale)
            for mode in (0, 1):
                out, lse = outs[mode]
                err = float(np.abs(out.cpu().numpy() - ref).max())
                err_l = float(np.abs(lse.cpu().numpy() - ref_lse).max())
                print(f"[loop live={live} step={t} mode={mode}] max|out-oracle|={err:.3e} "
                      f"max|lse-oracle|={err_l:.3e}", flush=True)
                assert np.isfinite(out.cpu().numpy()).all()
                assert err <= TOL and err_l <= TOL
                worst = max(worst, err, err_l)
    print(f"[loop live={live}] worst {worst:.3e}", flush=True)
