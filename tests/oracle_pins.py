"""Pins that tie the fp64 oracle to facts fixed independently of it.

Each ``pin_*`` raises ``AssertionError`` when the oracle disagrees with:
a 50-digit mpmath brute force written here from the definition (leaf sequence
= root-first concatenation of its path's segments, TreePO Sec. 2.3 segment
decomposition), closed forms (constant keys give the mean of V; a single key
gives that V; a zero query gives the mean of V), a library special case
(torch's scaled_dot_product_attention with grouped KV heads on a one-node
tree), invariants (identical paths give identical outputs; token order does
not matter), and the node-table closed forms of the full binary trees.
``test_oracle.py`` runs them; ``test_oracle_mutations.py`` plants mistakes in
the oracle and checks that some pin fails.
"""

from __future__ import annotations

import numpy as np

from oracle import attention as A
from oracle import cascade as C
from oracle import metadata as M
from workloads import build_call_log, node_kv_bits, query_bits
from workloads.data import bf16_round_bits, normal_bits

B = 64


def _bits(x) -> np.ndarray:
    return bf16_round_bits(np.asarray(x, dtype=np.float32))


def random_tiny_tree(seed: int, max_leaves: int = 6, max_tokens: int = 96):
    """A random small tree: (ops, leaves, rows).  Built without the oracle."""
    rng = np.random.default_rng(seed)
    ops, parent, length, children = [], [], [], []
    cap0 = int(rng.integers(1, 24))
    ops.append(("root", cap0)); parent.append(-1); length.append(0); children.append(0)
    ln = int(rng.integers(1, cap0 + 1))
    ops.append(("append", [0], [ln])); length[0] = ln
    tips = [0]
    total = {0: ln}
    while len(tips) < max_leaves and rng.random() < 0.85:
        p = tips[int(rng.integers(len(tips)))]
        if total[p] >= max_tokens - 1:
            break
        nkids = int(rng.integers(1, 3))
        cap = int(rng.integers(1, 20))
        first = len(parent)
        ops.append(("fork", p, nkids, cap))
        kids = list(range(first, first + nkids))
        for c in kids:
            parent.append(p); length.append(0); children.append(0)
        children[p] += nkids
        tips.remove(p)
        app_n, app_t = [], []
        for c in kids:
            t = int(rng.integers(0, min(cap, max_tokens - total[p]) + 1))
            length[c] = t
            total[c] = total[p] + t
            app_n.append(c); app_t.append(t)
            tips.append(c)
        ops.append(("append", app_n, app_t))
    leaves = [t for t in tips if total[t] > 0]
    if rng.random() < 0.5 and leaves:
        leaves.append(leaves[0])          # a duplicated leaf id
    rows = {i: length[i] for i in range(len(parent))}
    return ops, leaves, rows, parent


class _Log:
    def __init__(self, ops, leaves, rows):
        self.ops, self.leaves, self.rows, self.step_append = ops, leaves, rows, None


def _bf16_mp(bits: int):
    """The value of one bf16 bit pattern from its IEEE fields (sign, 8-bit
    biased exponent, 7-bit fraction), as an exact mpmath number: finite
    patterns only.  Independent of the oracle's widening."""
    import mpmath as mp
    b = int(bits) & 0xFFFF
    sign = -1 if b >> 15 else 1
    e, f = (b >> 7) & 0xFF, b & 0x7F
    assert e != 0xFF, "not a finite bf16"
    if e == 0:
        return sign * mp.ldexp(f, -133)          # subnormal: f * 2^-7 * 2^-126
    return sign * mp.ldexp(128 + f, e - 134)     # (1 + f/128) * 2^(e - 127)


def pin_bruteforce(seeds=(1, 2, 3, 4, 5, 6), hq=4, hkv=2, d=8, tol=1e-12):
    """50-digit brute force from the definition; the bf16 inputs are widened
    from their bit fields here, not by the oracle."""
    import mpmath as mp
    mp.mp.dps = 50
    for seed in seeds:
        ops, leaves, rows, parent = random_tiny_tree(seed)
        log = _Log(ops, leaves, rows)
        model = M.replay(log, B, 10_000, 10_000)
        data = {n: node_kv_bits(100 + seed, n, max(rows[n], 1), hkv, d) for n in rows}
        q = query_bits(100 + seed, 0, len(leaves), hq, d)
        scale = 1.0 / np.sqrt(d)
        out, lse = A.tree_decode(model, lambda n: data[n], leaves, q, scale)
        group = hq // hkv
        for pos, x in enumerate(leaves):
            path = []
            y = x
            while y != -1:
                path.append(y)
                y = parent[y]
            path.reverse()
            kseq, vseq = [], []
            for n in path:
                kb, vb = data[n]
                for t in range(rows[n]):
                    kseq.append([[_bf16_mp(kb[t, g, i]) for i in range(d)] for g in range(hkv)])
                    vseq.append([[_bf16_mp(vb[t, g, i]) for i in range(d)] for g in range(hkv)])
            qf = [[_bf16_mp(q[pos, h, i]) for i in range(d)] for h in range(hq)]
            for h in range(hq):
                g = h // group
                s = [mp.mpf(scale) * mp.fsum(qf[h][i] * k[g][i] for i in range(d)) for k in kseq]
                e = [mp.exp(si) for si in s]
                z = mp.fsum(e)
                for i in range(d):
                    o = mp.fsum(ei * v[g][i] for ei, v in zip(e, vseq)) / z
                    assert abs(float(o) - out[pos, h, i]) <= tol, (seed, pos, h, i)
                assert abs(float(mp.log(z)) - lse[pos, h]) <= tol, (seed, pos, h)


def _c1_model_and_data(kfun=None, vfun=None, seed=11, hq=4, hkv=2, d=16):
    log = build_call_log(1)
    model = M.replay(log, B, 10_000, 10_000)
    data = {}
    for n, r in log.rows.items():
        k, v = node_kv_bits(seed, n, r, hkv, d)
        if kfun is not None:
            k = kfun(n, r, k)
        if vfun is not None:
            v = vfun(n, r, v)
        data[n] = (k, v)
    return log, model, data


def pin_constant_keys(tol=1e-13):
    hq, hkv, d = 4, 2, 16
    kconst = _bits(np.random.default_rng(3).standard_normal((hkv, d)))
    log, model, data = _c1_model_and_data(
        kfun=lambda n, r, k: np.broadcast_to(kconst, k.shape).copy(), hq=hq, hkv=hkv, d=d)
    q = query_bits(11, 0, len(log.leaves), hq, d)
    out, _ = A.tree_decode(model, lambda n: data[n], log.leaves, q, 0.25)
    par = _parent_from_ops(log.ops)
    for pos, x in enumerate(log.leaves):
        # the leaf's values, collected by walking parents in the call log
        vs = []
        y = x
        while y != -1:
            vs.append(A.bf16_bits_to_f64(data[y][1][:log.rows[y]]))
            y = par[y]
        vall = np.concatenate(vs, axis=0)
        assert vall.shape[0] == 112
        for h in range(hq):
            np.testing.assert_allclose(out[pos, h], vall[:, h // (hq // hkv)].mean(axis=0),
                                       rtol=0, atol=tol)


def _parent_from_ops(ops):
    par, nid = {}, 0
    for op in ops:
        if op[0] == "root":
            par[nid] = -1; nid += 1
        elif op[0] == "fork":
            for _ in range(op[2]):
                par[nid] = op[1]; nid += 1
    return par


def pin_single_key():
    hq, hkv, d = 6, 3, 8
    model = M.TreeModel(B, 100, 100)
    r = model.new_root(1)
    model.append([r], [1])
    k, v = node_kv_bits(7, r, 1, hkv, d)
    q = query_bits(7, 0, 1, hq, d)
    out, lse = A.tree_decode(model, lambda n: (k, v), [r], q, 0.3)
    vf = A.bf16_bits_to_f64(v)
    kf = A.bf16_bits_to_f64(k)
    qf = A.bf16_bits_to_f64(q[0])
    for h in range(hq):
        g = h // (hq // hkv)
        assert np.array_equal(out[0, h], vf[0, g])
        assert abs(lse[0, h] - 0.3 * float(np.dot(qf[h], kf[0, g]))) <= 1e-14


def pin_zero_query(tol=1e-13):
    hq, hkv, d = 4, 2, 16
    log, model, data = _c1_model_and_data(hq=hq, hkv=hkv, d=d)
    q = np.zeros((len(log.leaves), hq, d), dtype=np.uint16)
    out, lse = A.tree_decode(model, lambda n: data[n], log.leaves, q, 0.125)
    par = _parent_from_ops(log.ops)
    for pos, x in enumerate(log.leaves):
        vs, y = [], x
        while y != -1:
            vs.append(A.bf16_bits_to_f64(data[y][1][:log.rows[y]]))
            y = par[y]
        vall = np.concatenate(vs)
        for h in range(hq):
            np.testing.assert_allclose(out[pos, h], vall[:, h // 2].mean(axis=0), rtol=0, atol=tol)
            assert abs(lse[pos, h] - np.log(vall.shape[0])) <= 1e-13


def pin_sdpa(tol=1e-12):
    import torch
    for (hq, hkv, d, L) in ((8, 2, 16, 37), (6, 3, 32, 130), (4, 4, 8, 5)):
        model = M.TreeModel(B, 100, 100)
        r = model.new_root(L)
        model.append([r], [L])
        k, v = node_kv_bits(21 + L, r, L, hkv, d)
        q = query_bits(21 + L, 0, 1, hq, d)
        scale = 0.7 / np.sqrt(d)
        out, _ = A.tree_decode(model, lambda n: (k, v), [r], q, scale)
        qt = torch.from_numpy(A.bf16_bits_to_f64(q[0]))[None, :, None, :]      # [1, Hq, 1, D]
        kt = torch.from_numpy(A.bf16_bits_to_f64(k)).permute(1, 0, 2)[None]    # [1, Hkv, L, D]
        vt = torch.from_numpy(A.bf16_bits_to_f64(v)).permute(1, 0, 2)[None]
        kt = kt.repeat_interleave(hq // hkv, dim=1)
        vt = vt.repeat_interleave(hq // hkv, dim=1)
        ref = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, scale=scale)
        np.testing.assert_allclose(out[0], ref[0, :, 0, :].numpy(), rtol=0, atol=tol)


def pin_identical_paths():
    hq, hkv, d = 4, 2, 16
    model = M.TreeModel(B, 100, 100)
    r = model.new_root(40)
    model.append([r], [40])
    a, b = model.fork(r, 2, 30)
    model.append([a, b], [30, 30])
    base = node_kv_bits(5, r, 40, hkv, d)
    kid = node_kv_bits(6, 0, 30, hkv, d)
    data = {r: base, a: kid, b: kid}
    q1 = query_bits(9, 0, 1, hq, d)
    q = np.concatenate([q1, q1, q1])
    out, lse = A.tree_decode(model, lambda n: data[n], [a, b, a], q, 0.2)
    assert np.array_equal(out[0], out[1]) and np.array_equal(out[0], out[2])
    assert np.array_equal(lse[0], lse[1])


def pin_permutation(tol=1e-12):
    hq, hkv, d, L = 4, 2, 16, 77
    k = A.bf16_bits_to_f64(normal_bits(1, 1, 0, (L, hkv, d)))
    v = A.bf16_bits_to_f64(normal_bits(1, 2, 0, (L, hkv, d)))
    q = A.bf16_bits_to_f64(normal_bits(1, 3, 0, (hq, d)))
    o1, l1 = A.attend(q, k, v, 0.25)
    perm = np.random.default_rng(0).permutation(L)
    o2, l2 = A.attend(q, k[perm], v[perm], 0.25)
    np.testing.assert_allclose(o1, o2, rtol=0, atol=tol)
    np.testing.assert_allclose(l1, l2, rtol=0, atol=tol)


def pin_cascade(tol=1e-12):
    """Per-node (and per-chunk) partials merged by the LSE rule == direct attention."""
    hq, hkv, d = 4, 2, 16
    log, model, data = _c1_model_and_data(hq=hq, hkv=hkv, d=d)
    q = query_bits(11, 0, len(log.leaves), hq, d)
    out, lse = A.tree_decode(model, lambda n: data[n], log.leaves, q, 0.25)
    rng = np.random.default_rng(0)
    for pos, x in enumerate(log.leaves):
        qf = A.bf16_bits_to_f64(q[pos])
        for h in range(hq):
            g = h // 2
            parts = [C.partial(qf[h], np.zeros((0, d)), np.zeros((0, d)), 0.25)]
            for n in model.chain(x):
                kf = A.bf16_bits_to_f64(data[n][0][:log.rows[n], g])
                vf = A.bf16_bits_to_f64(data[n][1][:log.rows[n], g])
                cut = sorted(rng.integers(0, kf.shape[0] + 1, size=2))
                for lo, hi in ((0, cut[0]), (cut[0], cut[1]), (cut[1], kf.shape[0])):
                    parts.append(C.partial(qf[h], kf[lo:hi], vf[lo:hi], 0.25))
            o, l = C.combine(parts)
            np.testing.assert_allclose(o, out[pos, h], rtol=0, atol=tol)
            assert abs(l - lse[pos, h]) <= tol


def pin_lse_logsumexp(tol=1e-12):
    from scipy.special import logsumexp
    hq, hkv, d, L = 4, 1, 8, 50
    k = A.bf16_bits_to_f64(normal_bits(4, 1, 0, (L, hkv, d)))
    v = A.bf16_bits_to_f64(normal_bits(4, 2, 0, (L, hkv, d)))
    q = A.bf16_bits_to_f64(normal_bits(4, 3, 0, (hq, d)))
    _, lse = A.attend(q, k, v, 0.5)
    for h in range(hq):
        assert abs(lse[h] - logsumexp(0.5 * (k[:, 0] @ q[h]))) <= tol


def pin_bf16_widening():
    """The oracle's bf16 -> fp64 widening against torch's own conversion on
    all 65,536 bit patterns (bit-exact on finite values, signed zeros
    included; the same class on infinities and NaNs), and against values
    written out from the IEEE bfloat16 format by hand."""
    import torch
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    with np.errstate(invalid="ignore"):
        mine = A.bf16_bits_to_f64(bits)
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).double().numpy()
    fin = np.isfinite(ref)
    assert fin.sum() == 65536 - 2 * 2 ** 7   # exponent 0xFF: 2 infinities + 254 NaNs
    assert np.array_equal(np.isfinite(mine), fin)
    assert np.array_equal(mine[fin].view(np.uint64), ref[fin].view(np.uint64))
    assert np.array_equal(np.isnan(mine), np.isnan(ref))
    inf = np.isinf(ref)
    assert inf.sum() == 2 and np.array_equal(mine[inf], ref[inf])
    hand = {0x3F80: 1.0, 0xC000: -2.0, 0x3E80: 0.25, 0x4049: 3.140625, 0x0000: 0.0, 0x8000: -0.0,
            0x0001: 2.0 ** -133, 0x807F: -127 * 2.0 ** -133, 0x0080: 2.0 ** -126,
            0x7F7F: (2 - 2 ** -7) * 2.0 ** 127, 0x7F80: np.inf, 0xFF80: -np.inf}
    got = A.bf16_bits_to_f64(np.array(list(hand), dtype=np.uint16))
    for b, g in zip(hand, got):
        want = hand[b]
        assert g == want and np.signbit(g) == np.signbit(want), (hex(b), g, want)
    with np.errstate(invalid="ignore"):
        assert np.isnan(A.bf16_bits_to_f64(np.array([0x7FC0, 0xFFC1, 0x7F81], dtype=np.uint16))).all()
    # finite patterns against the field decoding used by the brute force
    import mpmath as mp
    rng = np.random.default_rng(3)
    for b in rng.integers(0, 1 << 16, size=400):
        if (b >> 7) & 0xFF != 0xFF:
            assert mp.mpf(A.bf16_bits_to_f64(np.array([b], dtype=np.uint16))[0]) == _bf16_mp(b), hex(b)


def pin_positions_subset():
    """A decode restricted to some call positions (used on the large
    workloads) returns exactly those rows of the full decode, in the order
    asked, duplicates and repeats included."""
    hq, hkv, d = 6, 2, 16
    for seed in (3, 8, 12):
        ops, leaves, rows, _ = random_tiny_tree(seed, max_leaves=8)
        if not leaves:
            continue
        log = _Log(ops, leaves, rows)
        model = M.replay(log, B, 10_000, 10_000)
        data = {n: node_kv_bits(200 + seed, n, max(rows[n], 1), hkv, d) for n in rows}
        q = query_bits(200 + seed, 0, len(leaves), hq, d)
        out, lse = A.tree_decode(model, lambda n: data[n], leaves, q, 0.3)
        rng = np.random.default_rng(seed)
        pos = [int(p) for p in rng.integers(0, len(leaves), size=len(leaves) + 3)][::-1]
        o2, l2 = A.tree_decode(model, lambda n: data[n], leaves, q, 0.3, positions=pos)
        assert o2.shape == (len(pos), hq, d)
        assert np.array_equal(o2, out[pos]) and np.array_equal(l2, lse[pos])


# ---- node-table closed forms ----------------------------------------------

def pin_binary_heap_tiny():
    """Config 1 (level-order full binary tree): parent(n) = (n-1)//2, every node
    one 64-token block with id n, chain(x) = heap ancestors, starts 0,64,80,96."""
    log = build_call_log(1)
    m = M.replay(log, B, 10_000, 10_000)
    assert len(m.nodes) == 15
    assert log.leaves == list(range(7, 15))
    for n in range(15):
        rec = dict(zip(M.TreeModel.FIELDS, m.record(n)))
        assert rec["parent"] == ((n - 1) // 2 if n else -1)
        depth = int(np.floor(np.log2(n + 1)))
        assert rec["depth"] == depth
        assert rec["start"] == (0 if depth == 0 else 64 + 16 * (depth - 1))
        assert rec["len"] == (64 if n == 0 else 16)
        assert rec["block_begin"] == n and rec["n_blocks"] == 1 and rec["tree_id"] == 0
    for x in range(7, 15):
        anc = [x]
        while anc[-1]:
            anc.append((anc[-1] - 1) // 2)
        assert m.chain(x) == anc[::-1]
        assert m.leaf_blocks(x) == anc[::-1]
        assert m.chain_len(x) == 112
    ds = m.desc_sets(log.leaves)
    assert ds[0] == list(range(8))
    assert ds[1] == [0, 1, 2, 3] and ds[2] == [4, 5, 6, 7]
    for n in range(3, 7):
        assert ds[n] == [2 * (n - 3), 2 * (n - 3) + 1]
    for n in range(7, 15):
        assert ds[n] == [n - 7]


def pin_binary_heap_tiny_16_token_blocks():
    """Config 1 with 16-token blocks: the 64-token root reserves blocks 0-3,
    node n >= 1 (one 16-token segment) block n + 3; a leaf's blocks are its
    chain's runs, 4 + 3 = 7 of them for 112 tokens."""
    log = build_call_log(1)
    m = M.replay(log, 16, 10_000, 10_000)
    for n in range(15):
        rec = dict(zip(M.TreeModel.FIELDS, m.record(n)))
        assert (rec["block_begin"], rec["n_blocks"]) == ((0, 4) if n == 0 else (n + 3, 1))
    for x in range(7, 15):
        anc = [x]
        while anc[-1]:
            anc.append((anc[-1] - 1) // 2)
        want = [0, 1, 2, 3] + [a + 3 for a in anc[::-1][1:]]
        assert m.leaf_blocks(x) == want and len(want) == 7


def pin_single_tree_counts():
    """Config 2: 191 nodes, each 512 tokens = 8 blocks at 8n; 16 leaves with
    15-node chains of 7680 tokens; 97,792 unique tokens."""
    log = build_call_log(2)
    m = M.replay(log, B, 10_000, 10_000)
    assert len(m.nodes) == 191
    assert all(m.nodes[n]["block_begin"] == 8 * n and m.nodes[n]["n_blocks"] == 8 for n in range(191))
    assert sum(len(m.chain(x)) for x in log.leaves) == 240
    used = {n for x in log.leaves for n in m.chain(x)}
    assert sum(m.nodes[n]["len"] for n in used) == 97_792
    for x in log.leaves:
        ch = m.chain(x)
        assert len(ch) == 15 and m.chain_len(x) == 7680
        assert [m.nodes[n]["start"] for n in ch] == [512 * i for i in range(15)]
        assert m.leaf_blocks(x) == [8 * n + i for n in ch for i in range(8)]
    ds = m.desc_sets(log.leaves)
    sizes = sorted(len(v) for v in ds.values())
    assert sizes.count(16) == 1 and sizes.count(8) == 2 and sizes.count(4) == 4
    assert sizes.count(2) == 8 and sizes.count(1) == 176


def pin_long_context_counts():
    """Config 5: 2808 nodes, 256 leaves with 15-node chains of 16384 tokens
    after the fused one-token append; 2,883,584 unique tokens."""
    log = build_call_log(5)
    m = M.replay(log, B, 10 ** 6, 10 ** 6)
    assert len(m.nodes) == 2808 and len(log.leaves) == 256
    assert sum(len(m.chain(x)) for x in log.leaves) == 3840
    assert all(m.chain_len(x) == 16384 for x in log.leaves)
    used = {n for x in log.leaves for n in m.chain(x)}
    assert sum(m.nodes[n]["len"] for n in used) == 2_883_584
    assert len({m.nodes[x]["tree_id"] for x in log.leaves}) == 8


def pin_structure_invariants(cfgs=(1, 2, 3, 4, 5)):
    for c in cfgs:
        log = build_call_log(c)
        m = M.replay(log, B, 10 ** 7, 10 ** 7)
        nb = 0
        for n, nd in enumerate(m.nodes):
            assert nd["block_begin"] == nb
            nb += -(-nd["cap"] // B)
            assert nd["n_blocks"] == -(-nd["cap"] // B)
            p = nd["parent"]
            if p >= 0:
                assert p < n
                assert nd["depth"] == m.nodes[p]["depth"] + 1
                assert nd["start"] == m.nodes[p]["start"] + m.nodes[p]["len"]
                assert nd["tree_id"] == m.nodes[p]["tree_id"]
            assert 0 <= nd["len"] <= nd["cap"]
            assert nd["len"] == log.rows[n]


ALL_PINS = [pin_bf16_widening, pin_positions_subset, pin_bruteforce, pin_constant_keys, pin_single_key, pin_zero_query, pin_sdpa,
            pin_identical_paths, pin_permutation, pin_cascade, pin_lse_logsumexp,
            pin_binary_heap_tiny, pin_binary_heap_tiny_16_token_blocks, pin_single_tree_counts, pin_long_context_counts,
            pin_structure_invariants]
