"""Every status code forced from the host; a failing call changes no state.
The library's codes agree with the oracle model's on random op sequences."""

import numpy as np
import pytest

from oracle import metadata as M
from paper_2508_17445_amd import TreePOError
from paper_2508_17445_amd import treepo as T
from tests.lib_helpers import FAKE_POOL, ensure_lib, host_ctx


def _code(fn, *a):
    try:
        fn(*a)
    except TreePOError as e:
        return e.code
    return 0


def test_create_rejects_bad_configs():
    ensure_lib()
    from paper_2508_17445_amd import Context
    bad = [
        (dict(hq=6, hkv=4, d=64), T.EINVAL),
        (dict(hq=4, hkv=1, d=96), T.EUNSUPPORTED),
        (dict(hq=258, hkv=2, d=128), T.EUNSUPPORTED),
        (dict(hq=4, hkv=1, d=64, block_tokens=8), T.EUNSUPPORTED),
        (dict(hq=4, hkv=1, d=64, block_tokens=48), T.EUNSUPPORTED),
        (dict(hq=4, hkv=1, d=64, block_tokens=128), T.EUNSUPPORTED),
    ]
    for kw, code in bad:
        bt = kw.pop("block_tokens", 64)
        with pytest.raises(TreePOError) as e:
            Context(kw["hq"], kw["hkv"], kw["d"], 10, 10, FAKE_POOL, FAKE_POOL, bt)
        assert e.value.code == code
    with pytest.raises(TreePOError) as e:
        Context(4, 1, 64, 10, 10, 0, FAKE_POOL)
    assert e.value.code == T.EINVAL
    for bt in (16, 32, 64):  # the block sizes the pools take
        Context(4, 1, 64, 10, 10, FAKE_POOL, FAKE_POOL, bt).close()


def test_sixteen_token_blocks_keep_the_last_block_free():
    """With B = 16 a node's last 32-token tile may reach 16 rows past its
    blocks; the pool's last block is never reserved, so such a read stays in
    the pool.  B = 32 and 64 reserve every block."""
    ensure_lib()
    from paper_2508_17445_amd import Context
    for bt, usable in ((16, 9), (32, 10), (64, 10)):
        ctx = Context(4, 1, 64, 10, 10, FAKE_POOL, FAKE_POOL, bt)
        ctx.new_root(bt * (usable - 1))
        ctx.new_root(bt)
        with pytest.raises(TreePOError) as e:
            ctx.new_root(1)
        assert e.value.code == T.ENOMEM
        ctx.close()


def test_each_code_and_no_state_change():
    ctx = host_ctx(num_blocks=10, max_nodes=6)
    r = ctx.new_root(128)                                  # 2 blocks
    snap = ctx.export_nodes().copy()
    assert _code(ctx.new_root, 0) == T.EINVAL
    assert _code(ctx.fork, 7, 1, 64) == T.EINVAL
    assert _code(ctx.fork, r, 0, 64) == T.EINVAL
    assert _code(ctx.fork, r, 1, 0) == T.EINVAL
    assert _code(ctx.fork, r, 5, 64 * 2) == T.ENOMEM       # 10 blocks > 8 left
    assert _code(ctx.fork, r, 6, 1) == T.ENOMEM            # node table
    assert _code(ctx.kv_commit, [r], [129]) == T.EFULL
    assert _code(ctx.kv_commit, [r, r], [100, 29]) == T.EFULL
    assert _code(ctx.kv_commit, [r], [-1]) == T.EINVAL
    assert _code(ctx.kv_commit, [9], [1]) == T.EINVAL
    assert _code(ctx.workspace_size, [r]) == T.EEMPTY
    assert np.array_equal(ctx.export_nodes(), snap)
    ctx.kv_commit([r], [5])
    a, = ctx.fork(r, 1, 64)
    assert _code(ctx.kv_commit, [r], [1]) == T.EFROZEN
    assert _code(ctx.kv_commit, [a, r], [1, 1]) == T.EFROZEN   # whole call rejected
    assert ctx.export_nodes()[a][3] == 0
    assert _code(ctx.workspace_size, [a, 17]) == T.EINVAL
    assert _code(ctx.workspace_size, []) == T.EINVAL
    # decode: workspace is checked before any device work
    assert _code(ctx.tree_decode, [a], FAKE_POOL, 0.1, FAKE_POOL, None, None, 0) == T.EWORKSPACE
    assert _code(ctx.tree_decode, [a], None, 0.1, FAKE_POOL, None, FAKE_POOL, 1 << 30) == T.EINVAL
    for bad_scale in (0.0, -0.1, float("inf"), float("nan")):
        assert _code(ctx.tree_decode, [a], FAKE_POOL, bad_scale, FAKE_POOL, None, FAKE_POOL, 1 << 30) == T.EINVAL
        assert "scale" in ctx.lib.treepo_last_error(ctx.h).decode()
    # append with tokens but no K/V buffers
    assert _code(ctx.kv_append, [a], [1], None, None, 0) == T.EINVAL
    assert ctx.export_nodes()[a][3] == 0
    assert ctx.lib.treepo_last_error(ctx.h).decode() != ""


@pytest.mark.parametrize("seed", range(25))
def test_codes_match_oracle_on_random_ops(seed):
    rng = np.random.default_rng(seed)
    ctx = host_ctx(num_blocks=40, max_nodes=25)
    model = M.TreeModel(64, 40, 25)
    for _ in range(60):
        n = len(model.nodes)
        kind = rng.integers(5)
        if kind == 4 and n > 0:
            x = int(rng.integers(-1, n + 1))
            ln = model.nodes[x]["len"] if 0 <= x < n else 0
            offset = int(rng.choice([-1, 0, 64, 128, ln, int(rng.integers(0, max(ln, 1) + 1))]))
            args = (x, offset, int(rng.integers(-1, 3)), int(rng.integers(0, 200)))
            f_lib, f_ref = ctx.fork_at, model.fork_at
        elif kind == 0 or n == 0:
            cap = int(rng.integers(-1, 300))
            args = (cap,)
            f_lib, f_ref = ctx.new_root, model.new_root
        elif kind == 1:
            args = (int(rng.integers(-1, n + 1)), int(rng.integers(0, 4)), int(rng.integers(0, 200)))
            f_lib, f_ref = ctx.fork, model.fork
        else:
            k = int(rng.integers(1, 4))
            nodes = [int(x) for x in rng.integers(-1, n + 1, size=k)]
            ntok = [int(x) for x in rng.integers(-1, 80, size=k)]
            args = (nodes, ntok)
            f_lib, f_ref = ctx.kv_commit, model.append
        try:
            r_ref = f_ref(*args)
            c_ref = 0
        except M.TreeError as e:
            c_ref, r_ref = e.code, None
        try:
            r_lib = f_lib(*args)
            c_lib = 0
        except TreePOError as e:
            c_lib, r_lib = e.code, None
        assert c_lib == c_ref, (args, c_lib, c_ref)
        if c_ref == 0 and r_ref is not None:
            assert (list(r_lib) if isinstance(r_lib, tuple) else r_lib) == (list(r_ref) if isinstance(r_ref, tuple) else r_ref)
        ref = np.array([model.record(i) for i in range(len(model.nodes))], dtype=np.int32).reshape(-1, 8)
        assert np.array_equal(ctx.export_nodes().reshape(-1, 8), ref)


def test_advantage_codes():
    """treepo_tree_advantage validates before any device work; leaves need no tokens."""
    ctx = host_ctx()
    r = ctx.new_root(64)
    a, b = ctx.fork(r, 2, 64)
    nb = ctx.advantage_workspace_size([a, b])
    assert nb >= 256 and nb % 256 == 0
    assert _code(ctx.advantage_workspace_size, []) == T.EINVAL
    assert _code(ctx.advantage_workspace_size, [a, 99]) == T.EINVAL
    assert _code(ctx.tree_advantage, [a, b], FAKE_POOL, FAKE_POOL, FAKE_POOL, 2, 1 << 20) == T.EINVAL
    assert "weighting" in ctx.lib.treepo_last_error(ctx.h).decode()
    assert _code(ctx.tree_advantage, [a, b], None, FAKE_POOL, FAKE_POOL, 0, 1 << 20) == T.EINVAL
    assert _code(ctx.tree_advantage, [a, b], FAKE_POOL, None, FAKE_POOL, 0, 1 << 20) == T.EINVAL
    assert _code(ctx.tree_advantage, [a, 99], FAKE_POOL, FAKE_POOL, FAKE_POOL, 0, 1 << 20) == T.EINVAL
    assert _code(ctx.tree_advantage, [a, b], FAKE_POOL, FAKE_POOL, FAKE_POOL, 0, nb - 1) == T.EWORKSPACE
    assert _code(ctx.tree_advantage, [a, b], FAKE_POOL, FAKE_POOL, FAKE_POOL + 8, 0, nb) == T.EWORKSPACE
    assert _code(ctx.tree_advantage, [a, b], FAKE_POOL, FAKE_POOL, None, 0, nb) == T.EWORKSPACE


def test_prefill_codes_and_workspace_layout():
    """Prefill validation happens before any device work; the workspace holds
    32-byte work items (up to 128 tokens each), then 8-byte tile records of
    every chain (32 tokens each), the XCD schedule (8 int32 per slot), the
    append's 16-byte block pieces and its 8-byte length updates, each part at
    a 256-byte boundary."""
    ctx = host_ctx(num_blocks=40, max_nodes=8)
    r = ctx.new_root(300)
    # 3 items (10, 8 and 4 tiles: one XCD each, one slot); 10 tiles; 5 pieces; 1 update
    assert ctx.prefill_workspace_size([r], [300]) == 256 + 256 + 256 + 256 + 8
    assert ctx.prefill_workspace_size([r], [0]) == 256
    ctx.kv_commit([r], [100])
    a, b = ctx.fork(r, 2, 200)
    # a: chain 100 + 129 tokens -> 4 + 5 tiles, 2 items, 3 pieces.  b: 100 + 1 -> 4 + 1 tiles, 1 item, 1 piece
    assert ctx.prefill_workspace_size([a, b], [129, 1]) == 256 + 256 + 256 + 256 + 2 * 8
    snap = ctx.export_nodes().copy()
    F = FAKE_POOL
    assert _code(ctx.prefill, [a, a], [1, 1], F, F, F, 0.1, F, None, F, 1 << 20) == T.EINVAL   # a node twice
    assert "twice" in ctx.lib.treepo_last_error(ctx.h).decode()
    assert _code(ctx.prefill, [r], [1], F, F, F, 0.1, F, None, F, 1 << 20) == T.EFROZEN
    assert _code(ctx.prefill, [a], [201], F, F, F, 0.1, F, None, F, 1 << 20) == T.EFULL
    assert _code(ctx.prefill, [a], [1], None, F, F, 0.1, F, None, F, 1 << 20) == T.EINVAL
    assert _code(ctx.prefill, [a], [1], F, F, F, 0.1, None, None, F, 1 << 20) == T.EINVAL
    for bad_scale in (0.0, -1.0, float("inf"), float("nan")):
        assert _code(ctx.prefill, [a], [1], F, F, F, bad_scale, F, None, F, 1 << 20) == T.EINVAL
    need = ctx.prefill_workspace_size([a], [1])
    assert _code(ctx.prefill, [a], [1], F, F, F, 0.1, F, None, F, need - 1) == T.EWORKSPACE
    assert _code(ctx.prefill, [a], [1], F, F, F, 0.1, F, None, F + 16, need) == T.EWORKSPACE
    assert _code(ctx.prefill, [a], [1], F, F, F, 0.1, F, None, None, need) == T.EWORKSPACE
    assert np.array_equal(ctx.export_nodes(), snap)
    # nothing to prefill: no device work, no state change
    ctx.prefill([a, b], [0, 0], None, None, None, 0.1, None, None, None, 0)
    assert np.array_equal(ctx.export_nodes(), snap)


def test_noalloc_decode_rejects_plans_beyond_its_scratch():
    """The decode that allocates nothing keeps a plan image and the partial
    slots in 64 MiB of static device scratch; a decode needing more is
    EWORKSPACE (checked on the host, before any device call), with the bytes
    needed in the message."""
    from tests.lib_helpers import replay_host
    from workloads import CONFIGS, build_call_log
    c = CONFIGS[3]
    # the batch rollout's trees with twice its heads: ~125 MB of partial slots
    ctx = host_ctx(hq=2 * c.hq, hkv=2 * c.hkv, d=c.d)
    log = build_call_log(3)
    replay_host(ctx, log)
    assert ctx.workspace_size(log.leaves, 0) > 64 << 20
    with pytest.raises(TreePOError) as e:
        ctx.tree_decode_noalloc(log.leaves, FAKE_POOL, c.scale, FAKE_POOL, None)
    assert e.value.code == T.EWORKSPACE and "no-alloc scratch holds 67108864" in str(e.value)
    # the usual argument checks come first
    assert _code(ctx.tree_decode_noalloc, log.leaves, 0, c.scale, FAKE_POOL, None) == T.EINVAL
    assert _code(ctx.tree_decode_noalloc, log.leaves, FAKE_POOL, -1.0, FAKE_POOL, None) == T.EINVAL
    assert _code(ctx.tree_decode_noalloc, [10 ** 6], FAKE_POOL, c.scale, FAKE_POOL, None) == T.EINVAL
