"""Replays a workload call log into libtreepo on the GPU.

Input plumbing only: it creates the pools, issues the call log's
``new_root`` / ``fork`` / ``kv_append`` calls through the library binding with
the seeded bf16 rows of ``workloads.data``, and uploads the decode-step
queries.  Every computation is done by the library.
"""

from __future__ import annotations

import numpy as np

from .configs import CONFIGS, BLOCK_TOKENS, CallLog, Config, build_call_log
from .data import many_node_kv_bits, node_kv_bits, query_bits

# append calls are split so that one staging buffer stays below this many rows
_MAX_STAGE_ROWS = 1 << 16


def pool_blocks(log: CallLog, block_tokens: int = BLOCK_TOKENS) -> int:
    caps = [op[1] for op in log.ops if op[0] == "root"]
    caps += [op[3] for op in log.ops if op[0] == "fork" for _ in range(op[2])]
    caps += [op[4] for op in log.ops if op[0] == "fork_at" for _ in range(op[3])]
    return sum(-(-c // block_tokens) for c in caps)


class NodeData:
    """Lazily generated per-node K/V bit patterns: ``data(n)`` returns K, V
    whose row r is node n's r-th token (at least the rows it holds at decode).
    A tail cut from a node by ``fork_at`` reads that node's stream from the
    cut on."""

    def __init__(self, cfg: Config, log: CallLog):
        self.cfg, self.log = cfg, log
        self.src = getattr(log, "data_src", {}) or {}
        self.extra = getattr(log, "data_rows", {}) or {}
        self.cache: dict[int, tuple[np.ndarray, np.ndarray]] = {}

    def _rows(self, o: int) -> int:
        return self.extra.get(o, self.log.rows[o])

    def prefetch(self, nodes):
        todo = [o for o in dict.fromkeys(self.src.get(n, (n, 0))[0] for n in nodes) if o not in self.cache]
        if not todo:
            return
        res = many_node_kv_bits(self.cfg.seed, [(o, self._rows(o)) for o in todo], self.cfg.hkv, self.cfg.d)
        for o, kv in zip(todo, res):
            self.cache[o] = kv

    def __call__(self, n: int):
        o, first = self.src.get(n, (n, 0))
        if o not in self.cache:
            self.cache[o] = node_kv_bits(self.cfg.seed, o, self._rows(o), self.cfg.hkv, self.cfg.d)
        k, v = self.cache[o]
        return (k, v) if first == 0 else (k[first:], v[first:])

    def drop(self, nodes):
        for n in nodes:
            if n not in self.src and n not in self.extra:
                self.cache.pop(n, None)


class DeviceTree:
    """A workload's forest resident in GPU pools behind one library context."""

    def __init__(self, cfg_id: int | None = None, cfg: Config | None = None, log: CallLog | None = None,
                 device: str = "cuda", keep_host_data: bool = False, extra_blocks: int = 0,
                 apply_step_append: bool = True, live: bool = False):
        import torch
        from paper_2508_17445_amd import Context

        self.cfg = cfg if cfg is not None else CONFIGS[cfg_id]
        self.log = log if log is not None else build_call_log(cfg_id)
        self.device = device
        c = self.cfg
        # with 16-token blocks the library keeps the pool's last block free
        self.num_blocks = pool_blocks(self.log, c.block_tokens) + extra_blocks + (1 if c.block_tokens < 32 else 0)
        elems = c.hkv * self.num_blocks * c.block_tokens * c.d
        self.k_pool = torch.empty(elems, dtype=torch.bfloat16, device=device)
        self.v_pool = torch.empty(elems, dtype=torch.bfloat16, device=device)
        # live: node lengths on the device, plans reused across appends
        self.node_len = torch.zeros(max(self.log.n_nodes, 1), dtype=torch.int32, device=device) if live else None
        self.ctx = Context(c.hq, c.hkv, c.d, self.num_blocks, max(self.log.n_nodes, 1),
                           self.k_pool, self.v_pool, c.block_tokens, node_len=self.node_len)
        self.data = NodeData(c, self.log)
        self._len: dict[int, int] = {}
        self._replay(keep_host_data)
        self.leaves = list(self.log.leaves)
        self.q = self._to_dev(query_bits(c.seed, 0, len(self.leaves), c.hq, c.d))
        self.step_k = self.step_v = None
        if self.log.step_append is not None:
            nodes, ntok = self.log.step_append
            self.step_k, self.step_v = self._stage(nodes, ntok)
            if apply_step_append:
                self.step_append()

    # ---- helpers -------------------------------------------------------------
    def _to_dev(self, bits: np.ndarray):
        import torch
        t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).pin_memory()
        return t.to(self.device, non_blocking=True).view(torch.bfloat16)

    def _stage(self, nodes, ntok):
        self.data.prefetch(nodes)
        ks, vs = [], []
        cur = dict(self._len)
        for n, t in zip(nodes, ntok):
            lo = cur.get(n, 0)
            k, v = self.data(n)
            ks.append(k[lo:lo + t]); vs.append(v[lo:lo + t])
            cur[n] = lo + t
        return self._to_dev(np.concatenate(ks)), self._to_dev(np.concatenate(vs))

    def _replay(self, keep_host_data: bool):
        import torch
        for op in self.log.ops:
            if op[0] == "root":
                self.ctx.new_root(op[1])
            elif op[0] == "fork":
                self.ctx.fork(op[1], op[2], op[3])
            elif op[0] == "fork_at":
                x, off = op[1], op[2]
                _, t = self.ctx.fork_at(x, off, op[3], op[4])
                self._len[t] = self._len.get(x, 0) - off
                self._len[x] = off
            else:
                nodes, ntok = op[1], op[2]
                i = 0
                while i < len(nodes):
                    j, rows = i, 0
                    while j < len(nodes) and (j == i or rows + ntok[j] <= _MAX_STAGE_ROWS):
                        rows += ntok[j]
                        j += 1
                    sub_n, sub_t = nodes[i:j], ntok[i:j]
                    k, v = self._stage(sub_n, sub_t)
                    self.ctx.kv_append(sub_n, sub_t, k, v)
                    torch.cuda.synchronize()
                    for n, t in zip(sub_n, sub_t):
                        self._len[n] = self._len.get(n, 0) + t
                    if not keep_host_data:
                        self.data.drop([n for n in sub_n if self._len[n] == self.log.rows[n]
                                        and (self.log.step_append is None or n not in self.log.step_append[0])])
                    i = j

    def step_append(self):
        """The fused decode-step append (config 5): one token per leaf."""
        nodes, ntok = self.log.step_append
        self.ctx.kv_append(nodes, ntok, self.step_k, self.step_v)
        for n, t in zip(nodes, ntok):
            self._len[n] = self._len.get(n, 0) + t

    def outputs(self):
        import torch
        c = self.cfg
        out = torch.empty((len(self.leaves), c.hq, c.d), dtype=torch.float32, device=self.device)
        lse = torch.empty((len(self.leaves), c.hq), dtype=torch.float32, device=self.device)
        return out, lse

    def workspace(self, mode: int):
        import torch
        nbytes = self.ctx.workspace_size(self.leaves, mode)
        return torch.empty(max(nbytes, 256), dtype=torch.uint8, device=self.device)

    def decode(self, mode: int = 0, out=None, lse=None, ws=None):
        if out is None:
            out, lse = self.outputs()
        if ws is None:
            ws = self.workspace(mode)
        fn = self.ctx.tree_decode if mode == 0 else self.ctx.paged_decode_naive
        fn(self.leaves, self.q, self.cfg.scale, out, lse, ws)
        return out, lse

    def clone(self) -> "DeviceTree":
        """A replica with its own pools (device copy) and context (metadata replayed)."""
        import torch
        from paper_2508_17445_amd import Context
        r = object.__new__(DeviceTree)
        r.cfg, r.log, r.device, r.num_blocks = self.cfg, self.log, self.device, self.num_blocks
        r.k_pool = self.k_pool.clone()
        r.v_pool = self.v_pool.clone()
        c = self.cfg
        r.node_len = torch.zeros_like(self.node_len) if self.node_len is not None else None
        r.ctx = Context(c.hq, c.hkv, c.d, r.num_blocks, max(self.log.n_nodes, 1), r.k_pool, r.v_pool,
                        c.block_tokens, node_len=r.node_len)
        for op in self.log.ops:
            if op[0] == "root":
                r.ctx.new_root(op[1])
            elif op[0] == "fork":
                r.ctx.fork(op[1], op[2], op[3])
            elif op[0] == "fork_at":
                r.ctx.fork_at(op[1], op[2], op[3], op[4])
            else:
                r.ctx.kv_commit(op[1], op[2])
        r._len = dict(self._len)
        if self.log.step_append is not None and self._len.get(self.log.step_append[0][0], 0) == \
                self.log.rows[self.log.step_append[0][0]]:
            r.ctx.kv_commit(*self.log.step_append)
        r.data = self.data
        r.leaves = list(self.leaves)
        r.q = self.q.clone()
        r.step_k, r.step_v = self.step_k, self.step_v
        torch.cuda.synchronize()
        return r
