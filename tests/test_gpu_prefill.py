"""GPU parity of the prefill (treepo_prefill through the C-ABI) against the
fp64 oracle: causal attention of appended tokens over their chain.

Bar: max |out - oracle| <= 2e-3 and max |lse - oracle| <= 2e-3 over every
compared element.  Ragged prompt lengths around the 32-token tile and
the 128-token work item (1, 31, 32, 33, 127, 128, 129, 255, 256, 257, 513,
...), child segments that
attend to their whole chain, GQA groups 1 to 7, D = 64 and 128, the decode
after a prefill (the pool holds the prefilled rows), and the prompts of the
batch-rollout and long-context workloads at full size on sampled rows.
"""

from __future__ import annotations

import numpy as np
import pytest

from oracle import attention as A
from oracle import metadata as M
from oracle import prefill as PF
from workloads import CONFIGS, build_call_log, node_kv_bits, query_bits

TOL = 2e-3
B = 64

pytestmark = pytest.mark.gpu


class _Rig:
    """Pools, a context and the oracle model side by side."""

    def __init__(self, hq, hkv, d, seed, num_blocks, max_nodes=4096, live=False, bt=B):
        import torch
        from paper_2508_17445_amd import Context
        self.hq, self.hkv, self.d, self.seed = hq, hkv, d, seed
        self.scale = 1.0 / np.sqrt(d)
        elems = hkv * num_blocks * bt * d
        # pools filled with NaN bit patterns: rows past a node's length must never be read
        self.kp = torch.full((elems,), -1, dtype=torch.int16, device="cuda").view(torch.bfloat16)
        self.vp = torch.full((elems,), -1, dtype=torch.int16, device="cuda").view(torch.bfloat16)
        self.node_len = torch.zeros(max_nodes, dtype=torch.int32, device="cuda") if live else None
        self.ctx = Context(hq, hkv, d, num_blocks, max_nodes, self.kp, self.vp, bt, node_len=self.node_len)
        self.model = M.TreeModel(bt, num_blocks - (1 if bt < 32 else 0), max_nodes)
        self.kv = {}

    def dev(self, bits):
        import torch
        return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda().view(torch.bfloat16)

    def node_kv(self, n):
        return self.kv[n]

    def prefill(self, nodes, ntok, step):
        import torch
        ks, vs, qs = [], [], []
        for i, (x, t) in enumerate(zip(nodes, ntok)):
            k, v = node_kv_bits(self.seed, 10_000 * step + x, t, self.hkv, self.d)
            old = self.kv.get(x)
            self.kv[x] = (k, v) if old is None else (np.concatenate([old[0], k]), np.concatenate([old[1], v]))
            ks.append(k); vs.append(v)
            qs.append(query_bits(self.seed, 1000 * step + i, t, self.hq, self.d))
        kb, vb, qb = np.concatenate(ks), np.concatenate(vs), np.concatenate(qs)
        rows = int(sum(ntok))
        out = torch.full((rows, self.hq, self.d), float("nan"), dtype=torch.float32, device="cuda")
        lse = torch.full((rows, self.hq), float("nan"), dtype=torch.float32, device="cuda")
        ws = torch.empty(self.ctx.prefill_workspace_size(nodes, ntok), dtype=torch.uint8, device="cuda")
        self.ctx.prefill(nodes, ntok, self.dev(qb), self.dev(kb), self.dev(vb), self.scale, out, lse, ws)
        self.model.append(nodes, ntok)
        torch.cuda.synchronize()
        return qb, out.cpu().numpy(), lse.cpu().numpy()

    def check(self, nodes, ntok, qb, out, lse, tag, rows=None):
        ref, ref_l = PF.prefill(self.model, self.node_kv, nodes, ntok, qb, self.scale, rows=rows)
        o = out if rows is None else out[rows]
        l = lse if rows is None else lse[rows]
        err, err_l = float(np.abs(o - ref).max()), float(np.abs(l - ref_l).max())
        print(f"[prefill {tag}] rows={o.shape[0]} max|out-oracle|={err:.3e} max|lse-oracle|={err_l:.3e}", flush=True)
        assert np.isfinite(o).all() and np.isfinite(l).all()
        assert err <= TOL and err_l <= TOL


@pytest.mark.parametrize("hq,hkv,d,bt", [(28, 4, 128, 64), (4, 1, 64, 64), (8, 8, 128, 64), (12, 2, 64, 64),
                                         (28, 4, 128, 16), (4, 1, 64, 32)])
def test_ragged_prompts_then_segments(hq, hkv, d, bt):
    import torch
    lens = [1, 31, 32, 33, 64, 127, 128, 129, 300, 257, 255, 256, 513]
    print(f"[prefill ragged hq={hq} hkv={hkv} d={d} B={bt}]", flush=True)
    rig = _Rig(hq, hkv, d, 31 + d, num_blocks=400 * 64 // bt, bt=bt)
    roots = []
    for ln in lens:
        roots.append(rig.ctx.new_root(ln))
        assert rig.model.new_root(ln) == roots[-1]
    qb, out, lse = rig.prefill(roots, lens, 0)
    rig.check(roots, lens, qb, out, lse, "prompts")
    # the decode of every prompt reads what the prefill wrote
    q = query_bits(rig.seed, 77, len(roots), hq, d)
    o = torch.empty((len(roots), hq, d), dtype=torch.float32, device="cuda")
    l = torch.empty((len(roots), hq), dtype=torch.float32, device="cuda")
    ws = torch.empty(max(rig.ctx.workspace_size(roots, 0), 256), dtype=torch.uint8, device="cuda")
    rig.ctx.tree_decode(roots, rig.dev(q), rig.scale, o, l, ws)
    torch.cuda.synchronize()
    ref, ref_l = A.tree_decode(rig.model, rig.node_kv, roots, q, rig.scale)
    assert float(np.abs(o.cpu().numpy() - ref).max()) <= TOL
    assert float(np.abs(l.cpu().numpy() - ref_l).max()) <= TOL
    # child segments: each attends to its whole chain (prompt + own earlier tokens)
    kids = []
    for r in roots[:6]:
        c = rig.ctx.fork(r, 2, 200)
        assert rig.model.fork(r, 2, 200) == c
        kids += c
    seg = [1, 200, 33, 0, 129, 64, 2, 95, 160, 31, 128, 7]
    qb, out, lse = rig.prefill(kids, seg, 1)
    rig.check(kids, seg, qb, out, lse, "segments")
    # a second chunk on the same nodes continues the causal sequence
    more = [min(5, 200 - s) for s in seg]
    qb, out, lse = rig.prefill(kids, more, 2)
    rig.check(kids, more, qb, out, lse, "second chunk")


@pytest.mark.parametrize("cfg_id", [3, 5])
def test_workload_prompts_sampled(cfg_id):
    """Every prompt of the workload prefilled in one call; sampled rows."""
    import torch
    c = CONFIGS[cfg_id]
    log = build_call_log(cfg_id)
    plens = [op[1] for op in log.ops if op[0] == "root"]
    print(f"[prefill cfg{cfg_id}] prompts={len(plens)} tokens={sum(plens)}", flush=True)
    rig = _Rig(c.hq, c.hkv, c.d, c.seed, num_blocks=sum(-(-p // B) for p in plens) + 4, max_nodes=len(plens))
    roots = [rig.ctx.new_root(p) for p in plens]
    for p in plens:
        rig.model.new_root(p)
    qb, out, lse = rig.prefill(roots, plens, 0)
    rng = np.random.default_rng(cfg_id)
    starts = np.concatenate([[0], np.cumsum(plens)])
    rows = set()
    for i in rng.choice(len(plens), size=min(6, len(plens)), replace=False):
        b, e = int(starts[i]), int(starts[i + 1])
        rows |= {b, b + 1, e - 1, b + 127, b + 128, b + 255, b + 256} | {int(x) for x in rng.integers(b, e, size=4)}
    rows = sorted(r for r in rows if r < starts[-1])
    rig.check(roots, plens, qb, out, lse, f"cfg{cfg_id}", rows=rows)
    del rig
    torch.cuda.empty_cache()


def test_prefill_then_segment_decode_with_device_lengths():
    """Prompts prefilled, branches forked, a decode plan built once on device
    lengths; then branch segments prefilled in chunks (the append inside the
    prefill advances the device lengths) and the same plan decodes after
    every chunk."""
    import torch
    hq, hkv, d = 28, 4, 128
    rig = _Rig(hq, hkv, d, 555, num_blocks=200, live=True)
    lens = [200, 64, 33]
    roots = [rig.ctx.new_root(n) for n in lens]
    for n in lens:
        rig.model.new_root(n)
    qb, out, lse = rig.prefill(roots, lens, 0)
    rig.check(roots, lens, qb, out, lse, "live prompts")
    kids = []
    for r in roots:
        c = rig.ctx.fork(r, 2, 96)
        assert rig.model.fork(r, 2, 96) == c
        kids += c
    o = torch.empty((len(kids), hq, d), dtype=torch.float32, device="cuda")
    l = torch.empty((len(kids), hq), dtype=torch.float32, device="cuda")
    ws = torch.empty(max(rig.ctx.workspace_size(kids, 0), 256), dtype=torch.uint8, device="cuda")
    for step, chunk in enumerate(([1, 5, 40, 0, 17, 33], [31, 1, 24, 64, 30, 2], [0, 32, 32, 32, 0, 61])):
        qb, out, lse = rig.prefill(kids, chunk, step + 1)
        rig.check(kids, chunk, qb, out, lse, f"live chunk {step}")
        q = query_bits(rig.seed, 500 + step, len(kids), hq, d)
        rig.ctx.tree_decode(kids, rig.dev(q), rig.scale, o, l, ws)
        torch.cuda.synchronize()
        ref, ref_l = A.tree_decode(rig.model, rig.node_kv, kids, q, rig.scale)
        err = float(np.abs(o.cpu().numpy() - ref).max())
        print(f"[prefill live decode {step}] max|out-oracle|={err:.3e}", flush=True)
        assert err <= TOL and float(np.abs(l.cpu().numpy() - ref_l).max()) <= TOL


def test_prefill_after_a_cut():
    """A prompt cut inside (fork_at): its tail keeps growing (a prefill into
    the tail attends to the whole prompt), and the branches forked at the cut
    attend to the kept prefix only."""
    hq, hkv, d = 28, 4, 128
    rig = _Rig(hq, hkv, d, 777, num_blocks=200)
    r = rig.ctx.new_root(400)
    assert rig.model.new_root(400) == r
    qb, out, lse = rig.prefill([r], [300], 0)
    rig.check([r], [300], qb, out, lse, "cut: prompt")
    kids, t = rig.ctx.fork_at(r, 128, 2, 100)
    assert rig.model.fork_at(r, 128, 2, 100) == (kids, t)
    k, v = rig.kv[r]
    rig.kv[t] = (k[128:], v[128:])
    rig.kv[r] = (k[:128], v[:128])
    nodes, ntok = [t] + kids, [50, 30, 70]
    qb, out, lse = rig.prefill(nodes, ntok, 1)
    rig.check(nodes, ntok, qb, out, lse, "cut: tail and branches")


def test_prefill_is_deterministic():
    """The same call on two identical trees gives bitwise identical rows."""
    lens = [300, 129, 1]
    res = []
    for _ in range(2):
        rig = _Rig(28, 4, 128, 999, num_blocks=40)
        roots = [rig.ctx.new_root(n) for n in lens]
        for n in lens:
            rig.model.new_root(n)
        res.append(rig.prefill(roots, lens, 0)[1:])
    assert np.array_equal(res[0][0], res[1][0]) and np.array_equal(res[0][1], res[1][1])


def test_prefill_without_lse():
    """lse may be null: out is the same as with it."""
    import torch
    lens = [200, 33]
    outs = []
    for with_lse in (True, False):
        rig = _Rig(8, 2, 64, 4321, num_blocks=20)
        roots = [rig.ctx.new_root(n) for n in lens]
        k, v = zip(*(node_kv_bits(rig.seed, x, n, 2, 64) for x, n in zip(roots, lens)))
        q = query_bits(rig.seed, 0, sum(lens), 8, 64)
        out = torch.empty((sum(lens), 8, 64), dtype=torch.float32, device="cuda")
        lse = torch.empty((sum(lens), 8), dtype=torch.float32, device="cuda") if with_lse else None
        ws = torch.empty(rig.ctx.prefill_workspace_size(roots, lens), dtype=torch.uint8, device="cuda")
        rig.ctx.prefill(roots, lens, rig.dev(q), rig.dev(np.concatenate(k)), rig.dev(np.concatenate(v)), rig.scale,
                        out, lse, ws)
        torch.cuda.synchronize()
        outs.append(out.cpu().numpy())
    assert np.array_equal(outs[0], outs[1])
