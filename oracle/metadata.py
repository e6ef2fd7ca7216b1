"""Reference model of the segment-tree node table (pure Python).

TEST INFRASTRUCTURE ONLY (see the package docstring).

Rules, following TreePO Sec. 2.2 (tree vocabulary: the query is the root at
depth 0, segments of at most ``l`` tokens, a branching budget per node) and
Alg. 1 (paths are forked *before* each segment's inference; a generated
segment is appended to its path or the path stops):

* node ids are 0, 1, 2, ... in creation order; a fork's children take
  consecutive ids;
* a root has parent -1, depth 0, start 0 and ``tree_id`` equal to the number
  of roots created before it; a child has ``depth = parent.depth + 1``,
  ``start = parent.start + parent.len`` (its tokens follow the parent's) and
  the parent's ``tree_id``;
* a node that has children is frozen: nothing more is appended to it;
* every node reserves ``ceil(cap / B)`` pool blocks, contiguous, at creation;
  the first block id is the running total over all nodes created before it
  (one contiguous segment per node, the "contiguous segments" of the
  abstract); blocks are never freed;
* ``chain(x)`` is the root-first path to ``x``; the leaf's trajectory is the
  concatenation of its chain's segments (Sec. 2.3, segment decomposition);
* ``leaf_blocks(x)`` concatenates, along the chain, each node's first
  ``ceil(len / B)`` blocks;
* ``desc(n)`` for one decode call is the set of call positions whose chain
  contains ``n`` -- the nested subgroups G_j of Sec. 2.3 (Eq. groups).

Error codes mirror the library's C-ABI.
"""

from __future__ import annotations

OK = 0
EINVAL = -1
ENOMEM = -2
EFULL = -3
EFROZEN = -4
EEMPTY = -5


def _ceil_div(a: int, b: int) -> int:
    return -(-a // b)


class TreeError(Exception):
    def __init__(self, code: int, msg: str = ""):
        super().__init__(msg or str(code))
        self.code = code


class TreeModel:
    """Node table + block allocator, mutated by root / fork / append."""

    FIELDS = ("parent", "depth", "start", "len", "cap", "block_begin", "n_blocks", "tree_id")

    def __init__(self, block_tokens: int, num_blocks: int, max_nodes: int):
        if block_tokens <= 0 or num_blocks < 0 or max_nodes < 0:
            raise TreeError(EINVAL, "bad pool shape")
        self.B = block_tokens
        self.num_blocks = num_blocks
        self.max_nodes = max_nodes
        self.nodes: list[dict] = []
        self.n_children: list[int] = []
        self.next_block = 0
        self.n_roots = 0

    # ---- mutation -------------------------------------------------------
    def _reserve(self, count: int, cap: int) -> None:
        if cap <= 0:
            raise TreeError(EINVAL, "cap must be positive")
        if len(self.nodes) + count > self.max_nodes:
            raise TreeError(ENOMEM, "node table full")
        if self.next_block + count * _ceil_div(cap, self.B) > self.num_blocks:
            raise TreeError(ENOMEM, "pool blocks exhausted")

    def _make(self, parent: int, depth: int, start: int, cap: int, tree_id: int) -> int:
        nb = _ceil_div(cap, self.B)
        self.nodes.append(dict(parent=parent, depth=depth, start=start, len=0, cap=cap,
                               block_begin=self.next_block, n_blocks=nb, tree_id=tree_id))
        self.n_children.append(0)
        self.next_block += nb
        return len(self.nodes) - 1

    def new_root(self, cap: int) -> int:
        self._reserve(1, cap)
        nid = self._make(-1, 0, 0, cap, self.n_roots)
        self.n_roots += 1
        return nid

    def fork(self, parent: int, n: int, cap: int) -> list[int]:
        if not (0 <= parent < len(self.nodes)) or n < 1:
            raise TreeError(EINVAL, "bad fork")
        self._reserve(n, cap)
        p = self.nodes[parent]
        ids = [self._make(parent, p["depth"] + 1, p["start"] + p["len"], cap, p["tree_id"])
               for _ in range(n)]
        self.n_children[parent] += n
        return ids

    def fork_at(self, node: int, offset: int, n: int, cap: int):
        """Fork n children from node `node` after its first `offset` tokens: a
        fallback that branches inside a segment (Sec. 2.2 fallback at segment
        level; Sec. 4.2 "misaligned fallback" with a fallback granularity finer
        than the segment).  The node keeps tokens [0, offset); a new tail node
        (the next id) takes tokens [offset, len), the rest of the node's
        capacity and blocks, and the node's children, so every existing
        trajectory keeps its tokens; the tail's subtree moves one level down.
        Then the n children (consecutive ids, n may be 0) start after the
        kept prefix.  offset == len is a plain fork (tail -1); otherwise the
        offset must be a multiple of the block size (the tail starts on a
        block of its own, no KV is copied).  Returns (children, tail)."""
        if not (0 <= node < len(self.nodes)):
            raise TreeError(EINVAL, "unknown node")
        x = self.nodes[node]
        if not (0 <= offset <= x["len"]) or n < 0:
            raise TreeError(EINVAL, "bad offset or child count")
        if offset == x["len"]:
            return self.fork(node, n, cap), -1
        if offset % self.B:
            raise TreeError(EINVAL, "split offset not a multiple of the block size")
        if n > 0 and cap <= 0:
            raise TreeError(EINVAL, "cap must be positive")
        if len(self.nodes) + 1 + n > self.max_nodes:
            raise TreeError(ENOMEM, "node table full")
        if n > 0 and self.next_block + n * _ceil_div(cap, self.B) > self.num_blocks:
            raise TreeError(ENOMEM, "pool blocks exhausted")
        keep = offset // self.B
        tail = dict(parent=node, depth=x["depth"] + 1, start=x["start"] + offset, len=x["len"] - offset,
                    cap=x["cap"] - offset, block_begin=x["block_begin"] + keep, n_blocks=x["n_blocks"] - keep,
                    tree_id=x["tree_id"])
        self.nodes.append(tail)
        t = len(self.nodes) - 1
        self.n_children.append(self.n_children[node])
        moved = [c for c in range(len(self.nodes) - 1) if self.nodes[c]["parent"] == node]
        for c in moved:
            self.nodes[c]["parent"] = t
        stack = list(moved)
        while stack:
            c = stack.pop()
            self.nodes[c]["depth"] += 1
            stack += [d for d in range(len(self.nodes)) if self.nodes[d]["parent"] == c]
        x["len"] = offset
        x["cap"] = offset
        x["n_blocks"] = keep
        self.n_children[node] = 1
        kids = self.fork(node, n, cap) if n > 0 else []
        return kids, t

    def append(self, nodes, ntok) -> None:
        """Batched append: validated as a whole first, then applied in order."""
        if len(nodes) != len(ntok):
            raise TreeError(EINVAL, "length mismatch")
        pending: dict[int, int] = {}
        for n, t in zip(nodes, ntok):
            if not (0 <= n < len(self.nodes)) or t < 0:
                raise TreeError(EINVAL, "bad append")
            if self.n_children[n] > 0:
                raise TreeError(EFROZEN, "append to a node with children")
            pending[n] = pending.get(n, self.nodes[n]["len"]) + t
            if pending[n] > self.nodes[n]["cap"]:
                raise TreeError(EFULL, "append past cap")
        for n, ln in pending.items():
            self.nodes[n]["len"] = ln

    # ---- queries --------------------------------------------------------
    def record(self, n: int) -> list[int]:
        return [self.nodes[n][f] for f in self.FIELDS]

    def chain(self, x: int) -> list[int]:
        path = []
        while x != -1:
            path.append(x)
            x = self.nodes[x]["parent"]
        return path[::-1]

    def chain_len(self, x: int) -> int:
        return sum(self.nodes[n]["len"] for n in self.chain(x))

    def leaf_blocks(self, x: int) -> list[int]:
        out = []
        for n in self.chain(x):
            nd = self.nodes[n]
            out += list(range(nd["block_begin"], nd["block_begin"] + _ceil_div(nd["len"], self.B)))
        return out

    def desc_sets(self, leaves) -> dict[int, list[int]]:
        """node -> ascending call positions of the leaves whose chain contains it."""
        d: dict[int, list[int]] = {}
        for pos, x in enumerate(leaves):
            for n in self.chain(x):
                d.setdefault(n, []).append(pos)
        return dict(sorted(d.items()))

    def check_decode(self, leaves) -> None:
        for x in leaves:
            if not (0 <= x < len(self.nodes)):
                raise TreeError(EINVAL, "bad leaf id")
            if self.chain_len(x) == 0:
                raise TreeError(EEMPTY, "empty chain")


def replay(log, block_tokens: int, num_blocks: int, max_nodes: int,
           include_step_append: bool = True) -> TreeModel:
    """Apply a ``workloads.CallLog`` to a fresh model."""
    m = TreeModel(block_tokens, num_blocks, max_nodes)
    for op in log.ops:
        if op[0] == "root":
            m.new_root(op[1])
        elif op[0] == "fork":
            m.fork(op[1], op[2], op[3])
        elif op[0] == "fork_at":
            m.fork_at(op[1], op[2], op[3], op[4])
        elif op[0] == "append":
            m.append(op[1], op[2])
        else:
            raise ValueError(op[0])
    if include_step_append and log.step_append is not None:
        m.append(*log.step_append)
    return m


def pool_blocks_needed(log, block_tokens: int) -> int:
    caps = [op[1] for op in log.ops if op[0] == "root"]
    caps += [op[3] for op in log.ops if op[0] == "fork" for _ in range(op[2])]
    caps += [op[4] for op in log.ops if op[0] == "fork_at" for _ in range(op[3])]
    return sum(_ceil_div(c, block_tokens) for c in caps)
