"""The six synthetic segment-tree workloads and their call logs.

A call log is the sequence of library calls that builds a rollout forest the
way TreePO's tree sampler grows it (Alg. 1; Sec. 2.2 "Segment-level Tree
Sampling" and "Branching and Fallback"): every prompt is a root node, each
segment step forks the active paths *before* inference and then appends one
generated segment (at most ``l`` tokens) to every active path.  Steps are
level-synchronous across all prompts, as one ``Inference(P)`` call serves the
whole prompt queue.

Node ids follow the library's allocation rule (0, 1, 2, ... in creation order;
a fork's children take consecutive ids) so that ops can name the nodes they
touch.  The shapes are those of the paper's workloads: 7B-style GQA heads,
512-token segments, binary forks with up to 16 leaves (Sec. 3.1), 8x2048-token
evaluation trees (Table 2), random initial divergence and early stopping.
"""

from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Callable

from .data import structure_rng

BLOCK_TOKENS = 64


@dataclass
class CallLog:
    """Tree construction ops plus the decode step.

    ``ops`` items are ``("root", cap)``, ``("fork", parent, n_children, cap)``,
    ``("fork_at", node, offset, n_children, cap)`` (a fork after the first
    ``offset`` tokens of ``node``: a tail node takes the rest, then the
    children) or ``("append", nodes, ntok)`` (one batched append call).  The decode step
    is an optional fused append ``step_append`` (nodes, ntok) followed by a
    decode of ``leaves``.  ``rows[n]`` is node ``n``'s token count at decode
    time (after the fused append), which fixes how many K/V rows the data
    generator draws for it.  A tail made by ``fork_at`` holds rows of the
    node it was cut from: ``data_src[t] = (source node, first row)``, and a
    source node's stream is drawn with ``data_rows[n]`` rows when that
    exceeds ``rows[n]`` (the rows it held before a cut).
    """
    ops: list = field(default_factory=list)
    step_append: tuple | None = None
    leaves: list = field(default_factory=list)
    rows: dict = field(default_factory=dict)
    n_nodes: int = 0
    data_src: dict = field(default_factory=dict)
    data_rows: dict = field(default_factory=dict)


class _Builder:
    """Tracks ids, starts and lengths while emitting ops."""

    def __init__(self):
        self.log = CallLog()
        self.parent: list[int] = []
        self.start: list[int] = []
        self.len: list[int] = []
        self.cap: list[int] = []
        self.children: list[int] = []
        self.peak: list[int] = []
        self.src: dict[int, tuple[int, int]] = {}

    def _node(self, parent: int, start: int, cap: int) -> int:
        self.parent.append(parent); self.start.append(start); self.len.append(0)
        self.cap.append(cap); self.children.append(0); self.peak.append(0)
        return len(self.parent) - 1

    def root(self, cap: int) -> int:
        self.log.ops.append(("root", cap))
        return self._node(-1, 0, cap)

    def fork(self, p: int, n: int, cap: int) -> list[int]:
        self.log.ops.append(("fork", p, n, cap))
        return self._kids(p, n, cap)

    def _kids(self, p: int, n: int, cap: int) -> list[int]:
        self.children[p] += n
        return [self._node(p, self.start[p] + self.len[p], cap) for _ in range(n)]

    def fork_at(self, x: int, offset: int, n: int, cap: int):
        """Cut node x after `offset` tokens (a block multiple below its length):
        the tail takes the rest, x's children and blocks; then n children."""
        assert 0 <= offset < self.len[x] and offset % BLOCK_TOKENS == 0
        t = self._node(x, self.start[x] + offset, self.cap[x] - offset)
        self.len[t] = self.peak[t] = self.len[x] - offset
        self.children[t] = self.children[x]
        for c in range(t):
            if self.parent[c] == x:
                self.parent[c] = t
        o, first = self.src.get(x, (x, 0))
        self.src[t] = (o, first + offset)
        self.len[x] = self.cap[x] = offset
        self.children[x] = 1
        self.log.ops.append(("fork_at", x, offset, n, cap))
        return self._kids(x, n, cap), t

    def append(self, nodes: list[int], ntok: list[int]):
        for n, t in zip(nodes, ntok):
            assert self.len[n] + t <= self.cap[n] and self.children[n] == 0
            self.len[n] += t
            self.peak[n] = max(self.peak[n], self.len[n])
        if nodes:
            self.log.ops.append(("append", list(nodes), list(ntok)))

    def finish(self, leaves, step_append=None) -> CallLog:
        if step_append is not None:
            for n, t in zip(*step_append):
                self.len[n] += t
                self.peak[n] = max(self.peak[n], self.len[n])
            self.log.step_append = (list(step_append[0]), list(step_append[1]))
        self.log.leaves = list(leaves)
        self.log.rows = {i: self.len[i] for i in range(len(self.len))}
        self.log.n_nodes = len(self.len)
        need = {}
        for n in range(len(self.len)):
            o, first = self.src.get(n, (n, 0))
            need[o] = max(need.get(o, 0), first + self.peak[n])
        self.log.data_src = dict(self.src)
        self.log.data_rows = {o: r for o, r in need.items() if r > self.log.rows[o]}
        return self.log


def _binary_levels(b: _Builder, frontier: list[int], levels: int, seg: int,
                   fill: Callable[[int], int] | None = None) -> list[int]:
    for _ in range(levels):
        new = []
        for p in frontier:
            new += b.fork(p, 2, seg)
        b.append(new, [fill(n) if fill else seg for n in new])
        frontier = new
    return frontier


def gen_tiny(seed: int) -> CallLog:
    """One 64-token prompt, l=16, full binary forks at 3 boundaries: 8 leaves of 112."""
    b = _Builder()
    r = b.root(64)
    b.append([r], [64])
    leaves = _binary_levels(b, [r], 3, 16)
    return b.finish(leaves)


def gen_single_tree(seed: int) -> CallLog:
    """One 512-token prompt, l=512, binary forks at the first 4 boundaries
    (16 leaves), then unbranched segments to 7680 tokens per leaf."""
    b = _Builder()
    r = b.root(512)
    b.append([r], [512])
    front = _binary_levels(b, [r], 4, 512)
    while b.start[front[0]] + b.len[front[0]] < 7680:
        front = [b.fork(n, 1, 512)[0] for n in front]
        b.append(front, [512] * len(front))
    return b.finish(front)


def gen_batch_rollout(seed: int) -> CallLog:
    """64 prompts (256..1024 tokens) x 16 leaves, l=512, binary forks at the
    first 4 boundaries, leaf lengths uniform up to 8192 with a partial last
    segment."""
    rng = structure_rng(seed)
    seg, n_prompts = 512, 64
    plen = [int(x) for x in rng.integers(256, 1025, size=n_prompts)]
    b = _Builder()
    roots = [b.root(p) for p in plen]
    b.append(roots, plen)
    total = {}
    for i, p in enumerate(plen):
        lo = max(1024, p + 3 * seg + 1)
        total[i] = [int(x) for x in rng.integers(lo, 8193, size=16)]
    # three full binary levels, then the fourth level is sized by each leaf's total
    front = _binary_levels(b, roots, 3, seg)
    paths = []                       # (prompt, leaf index, current node)
    new = []
    for p in front:
        new += b.fork(p, 2, seg)
    # children are created prompt-major, 16 per prompt, in leaf order
    for k, n in enumerate(new):
        paths.append((k // 16, k % 16, n))
    b.append(new, [min(seg, total[i][j] - b.start[n]) for (i, j, n) in paths])
    active = [(i, j, n) for (i, j, n) in paths if b.start[n] + b.len[n] < total[i][j]]
    ends = {(i, j): n for (i, j, n) in paths}
    while active:
        nxt = []
        for (i, j, n) in active:
            c = b.fork(n, 1, seg)[0]
            nxt.append((i, j, c))
            ends[(i, j)] = c
        b.append([c for (_, _, c) in nxt],
                 [min(seg, total[i][j] - b.start[c]) for (i, j, c) in nxt])
        active = [(i, j, c) for (i, j, c) in nxt if b.start[c] + b.len[c] < total[i][j]]
    leaves = [ends[(i, j)] for i in range(n_prompts) for j in range(16)]
    return b.finish(leaves)


def gen_irregular(seed: int) -> CallLog:
    """32 prompts of 512 tokens, l=256; every active path forks into
    b ~ U{1,2,3,4} children (clipped to 32 leaves per prompt); each child stops
    early with p=0.2 after a random partial segment; paths end at 8192 tokens."""
    rng = structure_rng(seed)
    seg, n_prompts, max_leaves, max_len = 256, 32, 32, 8192
    b = _Builder()
    roots = [b.root(512) for _ in range(n_prompts)]
    b.append(roots, [512] * n_prompts)
    frontier = [[r] for r in roots]
    n_leaves = [1] * n_prompts
    while any(frontier):
        new_nodes, new_tok = [], []
        for p in range(n_prompts):
            nxt = []
            for n in sorted(frontier[p]):
                br = int(rng.integers(1, 5))
                br = min(br, max_leaves - n_leaves[p] + 1)
                kids = b.fork(n, br, seg)
                n_leaves[p] += br - 1
                for c in kids:
                    avail = min(seg, max_len - b.start[c])
                    if rng.random() < 0.2:
                        ln = int(rng.integers(1, avail + 1))
                    else:
                        ln = avail
                        if b.start[c] + ln < max_len:
                            nxt.append(c)
                    new_nodes.append(c); new_tok.append(ln)
            frontier[p] = nxt
        b.append(new_nodes, new_tok)
    leaves = [i for i in range(len(b.parent)) if b.children[i] == 0]
    return b.finish(leaves)


def gen_long_context(seed: int) -> CallLog:
    """8 prompts of 2048 tokens, l=1024, binary forks at the first 5 boundaries
    (32 leaves each), leaves grown to 16383 tokens; the decode step first
    appends one token to every leaf (to 16384) and then decodes."""
    seg = 1024
    b = _Builder()
    roots = [b.root(2048) for _ in range(8)]
    b.append(roots, [2048] * 8)
    front = _binary_levels(b, roots, 5, seg)
    while b.start[front[0]] + b.len[front[0]] + seg < 16384:
        front = [b.fork(n, 1, seg)[0] for n in front]
        b.append(front, [seg] * len(front))
    front = [b.fork(n, 1, seg)[0] for n in front]
    b.append(front, [seg - 1] * len(front))
    return b.finish(front, step_append=(front, [1] * len(front)))


def gen_misaligned_fallback(seed: int) -> CallLog:
    """32 prompts of 512 tokens, 7 segments of l=1024 (responses up to 7168
    tokens), width w=16, with a 512-token fallback (the misaligned setting of
    Sec. 4.2).  Level-synchronous steps: every active path forks into 2
    children while its prompt holds fewer than w live trajectories (1 after).
    Each child is pruned with p=0.2 after U[1, avail] tokens (an early stop:
    it stays in the forest but is no trajectory), ends with an answer with
    p=0.1 after U[1, avail] tokens, or takes the whole segment (finished at
    the length limit).  When a prompt has no active path and fewer than w
    trajectories, it falls back (Sec. 2.2): a random finished trajectory is
    re-forked into min(2, w - count) branches at a random 512-token boundary
    of its response; a boundary inside a 1024-token segment cuts that node
    (``fork_at``).  Every trajectory of the final forest is decoded."""
    rng = structure_rng(seed)
    seg, fb, plen, n_prompts, w = 1024, 512, 512, 32, 16
    p_prune, p_answer = 0.2, 0.1
    end = plen + 7 * seg
    b = _Builder()
    roots = [b.root(plen) for _ in range(n_prompts)]
    b.append(roots, [plen] * n_prompts)
    active = [[r] for r in roots]
    finished: list[list[int]] = [[] for _ in roots]
    count = [1] * n_prompts                       # active + finished trajectories
    while True:
        new_nodes, new_tok = [], []
        for p in range(n_prompts):
            if active[p]:
                grow = []
                for n in active[p]:
                    br = min(2 if count[p] < w else 1, w - count[p] + 1)
                    grow += b.fork(n, br, seg)
                    count[p] += br - 1
            elif count[p] < w and finished[p]:
                leaf = finished[p][int(rng.integers(len(finished[p])))]
                total = b.start[leaf] + b.len[leaf]
                pos = plen + fb * int(rng.integers(0, (total - 1 - plen) // fb + 1))
                x = leaf
                while b.start[x] > pos:
                    x = b.parent[x]
                br = min(2, w - count[p])
                if pos == b.start[x]:
                    grow = b.fork(b.parent[x], br, seg)
                else:
                    grow, t = b.fork_at(x, pos - b.start[x], br, seg)
                    if x == leaf:
                        finished[p][finished[p].index(leaf)] = t
                count[p] += br
            else:
                continue
            active[p] = []
            for c in grow:
                avail = min(seg, end - b.start[c])
                u = rng.random()
                if u < p_prune + p_answer:
                    ln = int(rng.integers(1, avail + 1))
                    if u < p_prune:
                        count[p] -= 1
                    else:
                        finished[p].append(c)
                else:
                    ln = avail
                    (active[p] if b.start[c] + ln < end else finished[p]).append(c)
                new_nodes.append(c)
                new_tok.append(ln)
        if not new_nodes:
            break
        b.append(new_nodes, new_tok)
    return b.finish([x for f in finished for x in f])


@dataclass(frozen=True)
class Config:
    name: str
    seed: int
    hq: int
    hkv: int
    d: int
    gen: Callable[[int], CallLog]
    block_tokens: int = BLOCK_TOKENS

    @property
    def scale(self) -> float:
        return 1.0 / math.sqrt(self.d)

    @property
    def group(self) -> int:
        return self.hq // self.hkv


CONFIGS = {
    1: Config("tiny-binary-8leaf", 1, 4, 1, 64, gen_tiny, block_tokens=16),  # one block per 16-token segment
    2: Config("single-tree-16leaf-7680", 2, 28, 4, 128, gen_single_tree),
    3: Config("batch-64x16-rollout", 3, 28, 4, 128, gen_batch_rollout),
    4: Config("irregular-32-prompt", 4, 28, 4, 128, gen_irregular),
    5: Config("long-context-8x32-16k", 5, 40, 8, 128, gen_long_context),
    6: Config("misaligned-fallback-32x16-7x1024", 6, 28, 4, 128, gen_misaligned_fallback),
}


def build_call_log(cfg_id: int) -> CallLog:
    cfg = CONFIGS[cfg_id]
    return cfg.gen(cfg.seed)
