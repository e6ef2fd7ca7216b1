"""Shared helpers for tests that load libtreepo.so (CPU-side calls only unless marked gpu)."""

from __future__ import annotations

import os

from oracle import metadata as M

FAKE_POOL = 0x10000  # device pointers are never dereferenced by host-side calls


def ensure_lib():
    from paper_2508_17445_amd.treepo import LIB_PATH, load_library
    if not os.path.exists(LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    return load_library()


def host_ctx(hq=4, hkv=1, d=64, num_blocks=1 << 20, max_nodes=1 << 20, block_tokens=64, live=False):
    ensure_lib()
    from paper_2508_17445_amd import Context
    return Context(hq, hkv, d, num_blocks, max_nodes, FAKE_POOL, FAKE_POOL + 64, block_tokens,
                   node_len=FAKE_POOL + 128 if live else None)


def replay_host(ctx, log, step_append=True):
    """Builds the log's tree in the library with metadata-only appends."""
    ids = []
    for op in log.ops:
        if op[0] == "root":
            ids.append(ctx.new_root(op[1]))
        elif op[0] == "fork":
            ids += ctx.fork(op[1], op[2], op[3])
        elif op[0] == "fork_at":
            kids, t = ctx.fork_at(op[1], op[2], op[3], op[4])
            ids += [t] + kids
        else:
            ctx.kv_commit(op[1], op[2])
    if step_append and log.step_append is not None:
        ctx.kv_commit(*log.step_append)
    return ids


def oracle_model(log, num_blocks=1 << 20, max_nodes=1 << 20, block_tokens=64):
    return M.replay(log, block_tokens, num_blocks, max_nodes)
