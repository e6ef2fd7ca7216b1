"""ctypes binding of libtreepo.so (argument marshalling only).

Every function here forwards to the C-ABI declared in ``include/treepo.h``
with the same name; device buffers are passed as raw device addresses
(``int``) or as torch tensors, streams as raw ``hipStream_t`` handles or torch
streams.  All computation happens in the library's HIP kernels; if the shared
library is missing this module raises instead of computing anything itself.
"""

from __future__ import annotations

import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
# TREEPO_LIBRARY selects another build of the same C-ABI (the host-sanitizer
# build in the CPU tests); by default the in-tree libtreepo.so is loaded.
LIB_PATH = os.environ.get("TREEPO_LIBRARY") or os.path.join(HERE, "libtreepo.so")

OK, EINVAL, ENOMEM, EFULL, EFROZEN, EEMPTY, EWORKSPACE, EHIP, EUNSUPPORTED = 0, -1, -2, -3, -4, -5, -6, -7, -8
MODE_TREE, MODE_NAIVE = 0, 1
KERNEL_APPEND, KERNEL_PARTIAL, KERNEL_COMBINE, KERNEL_ADVANTAGE, KERNEL_PREFILL = 0, 1, 2, 3, 4
ADV_MEAN, ADV_SIZE_WEIGHTED = 0, 1
NODE_FIELDS = ("parent", "depth", "start", "len", "cap", "block_begin", "n_blocks", "tree_id")
BLOCK_TOKENS = 64
PIECE_FIELDS = 16
TILE_FIELDS = 4

_i32 = ctypes.c_int32
_i64 = ctypes.c_int64
_p = ctypes.c_void_p
_pi32 = ctypes.POINTER(ctypes.c_int32)
_pi64 = ctypes.POINTER(ctypes.c_int64)


class TreePOError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{msg} (status {code})")
        self.code = code


class Config(ctypes.Structure):
    _fields_ = [("num_q_heads", _i32), ("num_kv_heads", _i32), ("head_dim", _i32),
                ("block_tokens", _i32), ("num_blocks", _i64), ("max_nodes", _i32),
                ("reserved", _i32), ("k_pool", _p), ("v_pool", _p), ("node_len", _p)]


_lib = None


def load_library(path: str = LIB_PATH):
    """Loads the shared library (once).  Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built; run __graft_entry__.build()")
    lib = ctypes.CDLL(path)
    sig = {
        "treepo_create": (_i32, [ctypes.POINTER(Config), ctypes.POINTER(_p)]),
        "treepo_destroy": (_i32, [_p]),
        "treepo_set_device_shape": (_i32, [_p, _i32, _i32]),
        "treepo_new_root": (_i32, [_p, _i32, _pi32]),
        "treepo_fork": (_i32, [_p, _i32, _i32, _i32, _pi32]),
        "treepo_fork_at": (_i32, [_p, _i32, _i32, _i32, _i32, _pi32, _pi32]),
        "treepo_kv_append": (_i32, [_p, _i32, _pi32, _pi32, _p, _p, _p]),
        "treepo_kv_slots": (_i32, [_p, _i32, _pi32, _pi32, _pi64]),
        "treepo_kv_commit": (_i32, [_p, _i32, _pi32, _pi32]),
        "treepo_decode_workspace_size": (_i32, [_p, _i32, _pi32, _i32, ctypes.POINTER(ctypes.c_size_t)]),
        "treepo_tree_decode": (_i32, [_p, _i32, _pi32, _p, ctypes.c_float, _p, _p, _p, ctypes.c_size_t, _p]),
        "treepo_paged_decode_naive": (_i32, [_p, _i32, _pi32, _p, ctypes.c_float, _p, _p, _p, ctypes.c_size_t, _p]),
        "treepo_tree_decode_noalloc": (_i32, [_p, _i32, _pi32, _p, ctypes.c_float, _p, _p, _p]),
        "treepo_num_nodes": (_i32, [_p, _pi32]),
        "treepo_export_nodes": (_i32, [_p, _pi32, _i32, _pi32]),
        "treepo_export_chains": (_i32, [_p, _i32, _pi32, _pi32, _pi32, _pi32, _pi32, _pi32, _pi32]),
        "treepo_export_desc": (_i32, [_p, _i32, _pi32, _pi32, _pi32, _pi32, _pi32, _pi32]),
        "treepo_export_plan": (_i32, [_p, _i32, _pi32, _i32, _pi32, _pi32, _pi32, _pi32, _pi32, _pi32, _pi32]),
        "treepo_export_blocks": (_i32, [_p, _i32, _pi32, _i32, _pi32, _pi32, _pi32]),
        "treepo_set_profiling": (_i32, [_p, _i32]),
        "treepo_profile_read": (_i32, [_p, _i32, ctypes.POINTER(ctypes.c_double), _pi64]),
        "treepo_strerror": (ctypes.c_char_p, [_i32]),
        "treepo_last_error": (ctypes.c_char_p, [_p]),
        "treepo_branch_budget": (_i32, [_i32, ctypes.POINTER(ctypes.c_float), _i32, _i32, ctypes.c_float, _pi32]),
        "treepo_advantage_workspace_size": (_i32, [_p, _i32, _pi32, ctypes.POINTER(ctypes.c_size_t)]),
        "treepo_tree_advantage": (_i32, [_p, _i32, _pi32, _p, _i32, _p, _p, ctypes.c_size_t, _p]),
        "treepo_prefill_workspace_size": (_i32, [_p, _i32, _pi32, _pi32, ctypes.POINTER(ctypes.c_size_t)]),
        "treepo_prefill": (_i32, [_p, _i32, _pi32, _pi32, _p, _p, _p, ctypes.c_float, _p, _p, _p, ctypes.c_size_t,
                                  _p]),
        "treepo_bench_copy": (_i32, [_p, _p, ctypes.c_size_t, _p]),
        "treepo_bench_read": (_i32, [_p, ctypes.c_size_t, _p, _p]),
        "treepo_bench_stream": (_i32, [_p, ctypes.c_size_t, _p, _i32, _i32, _p]),
        "treepo_bench_overlap": (_i32, [_i32, _i32, _i32, _p, _p, _p]),
    }
    for name, (res, args) in sig.items():
        if name.startswith("treepo_bench_") and not hasattr(lib, name):
            continue  # measurement probes are absent from host-only builds
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    _lib = lib
    return lib


def _arr32(xs) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(xs, dtype=np.int32).reshape(-1))


def _ptr32(a: np.ndarray):
    return a.ctypes.data_as(_pi32)


def _dev(x) -> int | None:
    """Device address of a torch tensor, an int address, or None."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return int(x.data_ptr())


def _stream(s) -> int | None:
    if s is None:
        try:
            import torch
            return int(torch.cuda.current_stream().cuda_stream)
        except Exception:
            return None
    if isinstance(s, int):
        return s
    return int(s.cuda_stream)


class Context:
    """One segment-tree KV cache over caller-owned K/V pools."""

    def __init__(self, num_q_heads: int, num_kv_heads: int, head_dim: int, num_blocks: int,
                 max_nodes: int, k_pool, v_pool, block_tokens: int = BLOCK_TOKENS, node_len=None):
        self.lib = load_library()
        self.cfg = Config(num_q_heads, num_kv_heads, head_dim, block_tokens, num_blocks,
                          max_nodes, 0, _dev(k_pool), _dev(v_pool),
                          _dev(node_len) if node_len is not None else None)
        self._keep = (k_pool, v_pool, node_len)
        h = _p()
        st = self.lib.treepo_create(ctypes.byref(self.cfg), ctypes.byref(h))
        if st != OK:
            raise TreePOError(st, "treepo_create: " + self.lib.treepo_strerror(st).decode())
        self.h = h

    def close(self):
        if getattr(self, "h", None):
            self.lib.treepo_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def _check(self, st: int, what: str):
        if st != OK:
            msg = self.lib.treepo_last_error(self.h).decode() or self.lib.treepo_strerror(st).decode()
            raise TreePOError(st, f"{what}: {msg}")

    def set_device_shape(self, compute_units: int, xcds: int):
        self._check(self.lib.treepo_set_device_shape(self.h, compute_units, xcds), "treepo_set_device_shape")

    # ---- tree --------------------------------------------------------------
    def new_root(self, cap: int) -> int:
        n = _i32()
        self._check(self.lib.treepo_new_root(self.h, cap, ctypes.byref(n)), "treepo_new_root")
        return n.value

    def fork(self, parent: int, n_children: int, child_cap: int) -> list[int]:
        out = np.zeros(max(n_children, 1), dtype=np.int32)
        self._check(self.lib.treepo_fork(self.h, parent, n_children, child_cap, _ptr32(out)), "treepo_fork")
        return [int(x) for x in out[:n_children]]

    def fork_at(self, node: int, offset: int, n_children: int, child_cap: int):
        """Fork after the first `offset` tokens of `node`: (children, tail id or -1)."""
        out = np.zeros(max(n_children, 1), dtype=np.int32)
        tail = _i32()
        self._check(self.lib.treepo_fork_at(self.h, node, offset, n_children, child_cap, _ptr32(out),
                                            ctypes.byref(tail)), "treepo_fork_at")
        return [int(x) for x in out[:n_children]], tail.value

    def kv_append(self, nodes, ntok, k, v, stream=None):
        nd, nt = _arr32(nodes), _arr32(ntok)
        self._check(self.lib.treepo_kv_append(self.h, len(nd), _ptr32(nd), _ptr32(nt), _dev(k), _dev(v),
                                              _stream(stream)), "treepo_kv_append")

    def kv_slots(self, nodes, ntok) -> np.ndarray:
        nd, nt = _arr32(nodes), _arr32(ntok)
        rows = np.zeros(max(int(nt.sum()), 1), dtype=np.int64)
        self._check(self.lib.treepo_kv_slots(self.h, len(nd), _ptr32(nd), _ptr32(nt),
                                             rows.ctypes.data_as(_pi64)), "treepo_kv_slots")
        return rows[:int(nt.sum())]

    def kv_commit(self, nodes, ntok):
        nd, nt = _arr32(nodes), _arr32(ntok)
        self._check(self.lib.treepo_kv_commit(self.h, len(nd), _ptr32(nd), _ptr32(nt)), "treepo_kv_commit")

    # ---- decode ------------------------------------------------------------
    def workspace_size(self, leaves, mode: int = MODE_TREE) -> int:
        lv = _arr32(leaves)
        b = ctypes.c_size_t()
        self._check(self.lib.treepo_decode_workspace_size(self.h, len(lv), _ptr32(lv), mode, ctypes.byref(b)),
                    "treepo_decode_workspace_size")
        return b.value

    def _decode(self, fn, name, leaves, q, scale, out, lse, workspace, ws_bytes, stream):
        lv = _arr32(leaves)
        if ws_bytes is None:
            ws_bytes = int(workspace.numel() * workspace.element_size())
        self._check(fn(self.h, len(lv), _ptr32(lv), _dev(q), ctypes.c_float(scale), _dev(out), _dev(lse),
                       _dev(workspace), ws_bytes, _stream(stream)), name)

    def tree_decode(self, leaves, q, scale, out, lse, workspace, ws_bytes=None, stream=None):
        self._decode(self.lib.treepo_tree_decode, "treepo_tree_decode", leaves, q, scale, out, lse,
                     workspace, ws_bytes, stream)

    def paged_decode_naive(self, leaves, q, scale, out, lse, workspace, ws_bytes=None, stream=None):
        self._decode(self.lib.treepo_paged_decode_naive, "treepo_paged_decode_naive", leaves, q, scale,
                     out, lse, workspace, ws_bytes, stream)

    def tree_decode_noalloc(self, leaves, q, scale, out, lse, stream=None):
        lv = _arr32(leaves)
        self._check(self.lib.treepo_tree_decode_noalloc(self.h, len(lv), _ptr32(lv), _dev(q), ctypes.c_float(scale),
                                                        _dev(out), _dev(lse), _stream(stream)),
                    "treepo_tree_decode_noalloc")

    # ---- export ------------------------------------------------------------
    def num_nodes(self) -> int:
        n = _i32()
        self._check(self.lib.treepo_num_nodes(self.h, ctypes.byref(n)), "treepo_num_nodes")
        return n.value

    def export_nodes(self) -> np.ndarray:
        n = self.num_nodes()
        rec = np.zeros((max(n, 1), len(NODE_FIELDS)), dtype=np.int32)
        got = _i32()
        self._check(self.lib.treepo_export_nodes(self.h, _ptr32(rec), n, ctypes.byref(got)), "treepo_export_nodes")
        return rec[:n]

    def export_chains(self, leaves):
        lv = _arr32(leaves)
        tc, tb = _i32(), _i32()
        z = ctypes.POINTER(ctypes.c_int32)()
        self._check(self.lib.treepo_export_chains(self.h, len(lv), _ptr32(lv), z, z, z, z,
                                                  ctypes.byref(tc), ctypes.byref(tb)), "treepo_export_chains")
        co = np.zeros(len(lv) + 1, np.int32); cn = np.zeros(max(tc.value, 1), np.int32)
        bo = np.zeros(len(lv) + 1, np.int32); bl = np.zeros(max(tb.value, 1), np.int32)
        self._check(self.lib.treepo_export_chains(self.h, len(lv), _ptr32(lv), _ptr32(co), _ptr32(cn),
                                                  _ptr32(bo), _ptr32(bl), ctypes.byref(tc), ctypes.byref(tb)),
                    "treepo_export_chains")
        return co, cn[:tc.value], bo, bl[:tb.value]

    def export_desc(self, leaves):
        lv = _arr32(leaves)
        nn, tot = _i32(), _i32()
        z = ctypes.POINTER(ctypes.c_int32)()
        self._check(self.lib.treepo_export_desc(self.h, len(lv), _ptr32(lv), z, z, z, ctypes.byref(nn),
                                                ctypes.byref(tot)), "treepo_export_desc")
        nodes = np.zeros(max(nn.value, 1), np.int32); off = np.zeros(nn.value + 1, np.int32)
        desc = np.zeros(max(tot.value, 1), np.int32)
        self._check(self.lib.treepo_export_desc(self.h, len(lv), _ptr32(lv), _ptr32(nodes), _ptr32(off),
                                                _ptr32(desc), ctypes.byref(nn), ctypes.byref(tot)),
                    "treepo_export_desc")
        return nodes[:nn.value], off, desc[:tot.value]

    def export_plan(self, leaves, mode: int = MODE_TREE):
        """(pieces [n, PIECE_FIELDS], rowsets, tiles [m, TILE_FIELDS], n_streams)."""
        lv = _arr32(leaves)
        ni, nr, nt, ns = _i32(), _i32(), _i32(), _i32()
        z = ctypes.cast(None, _pi32)
        self._check(self.lib.treepo_export_plan(self.h, len(lv), _ptr32(lv), mode, z, z, z, ctypes.byref(ni),
                                                ctypes.byref(nr), ctypes.byref(nt), ctypes.byref(ns)),
                    "treepo_export_plan")
        pieces = np.zeros((max(ni.value, 1), PIECE_FIELDS), np.int32)
        rowsets = np.zeros(max(nr.value, 1), np.int32)
        tiles = np.zeros((max(nt.value, 1), TILE_FIELDS), np.int32)
        self._check(self.lib.treepo_export_plan(self.h, len(lv), _ptr32(lv), mode, _ptr32(pieces), _ptr32(rowsets),
                                                _ptr32(tiles), ctypes.byref(ni), ctypes.byref(nr), ctypes.byref(nt),
                                                ctypes.byref(ns)),
                    "treepo_export_plan")
        return pieces[:ni.value], rowsets[:nr.value], tiles[:nt.value], ns.value

    def export_blocks(self, leaves, mode: int = MODE_TREE):
        """Stream blocks as the kernel reads them: int32 [n_streams, block_ints]."""
        lv = _arr32(leaves)
        bi, ns = _i32(), _i32()
        self._check(self.lib.treepo_export_blocks(self.h, len(lv), _ptr32(lv), mode, ctypes.cast(None, _pi32),
                                                  ctypes.byref(bi), ctypes.byref(ns)), "treepo_export_blocks")
        out = np.zeros((max(ns.value, 1), max(bi.value, 1)), np.int32)
        self._check(self.lib.treepo_export_blocks(self.h, len(lv), _ptr32(lv), mode, _ptr32(out), ctypes.byref(bi),
                                                  ctypes.byref(ns)), "treepo_export_blocks")
        return out[:ns.value]

    # ---- TreePO advantage --------------------------------------------------
    def advantage_workspace_size(self, leaves) -> int:
        lv = _arr32(leaves)
        n = ctypes.c_size_t()
        self._check(self.lib.treepo_advantage_workspace_size(self.h, len(lv), _ptr32(lv), ctypes.byref(n)),
                    "treepo_advantage_workspace_size")
        return n.value

    def tree_advantage(self, leaves, rewards, adv, workspace, weighting: int = 0, ws_bytes=None, stream=None):
        """adv[p] = TreePO advantage of call position p (rewards, adv: device fp32)."""
        lv = _arr32(leaves)
        nb = int(workspace.numel() * workspace.element_size()) if ws_bytes is None else ws_bytes
        self._check(self.lib.treepo_tree_advantage(self.h, len(lv), _ptr32(lv), _dev(rewards), weighting, _dev(adv),
                                                   _dev(workspace), nb, _stream(stream)), "treepo_tree_advantage")

    # ---- prefill -------------------------------------------------------------
    def prefill_workspace_size(self, nodes, ntok) -> int:
        nd, nt = _arr32(nodes), _arr32(ntok)
        n = ctypes.c_size_t()
        self._check(self.lib.treepo_prefill_workspace_size(self.h, len(nd), _ptr32(nd), _ptr32(nt), ctypes.byref(n)),
                    "treepo_prefill_workspace_size")
        return n.value

    def prefill(self, nodes, ntok, q, k, v, scale, out, lse, workspace, ws_bytes=None, stream=None):
        """Append ntok[i] tokens to nodes[i] and write their causal attention
        over the chain (q, k, v, out, lse: device tensors packed in call order)."""
        nd, nt = _arr32(nodes), _arr32(ntok)
        nb = int(workspace.numel() * workspace.element_size()) if ws_bytes is None else ws_bytes
        self._check(self.lib.treepo_prefill(self.h, len(nd), _ptr32(nd), _ptr32(nt), _dev(q), _dev(k), _dev(v),
                                            float(scale), _dev(out), _dev(lse), _dev(workspace), nb, _stream(stream)),
                    "treepo_prefill")

    # ---- timing ------------------------------------------------------------
    def set_profiling(self, enable: bool):
        self._check(self.lib.treepo_set_profiling(self.h, 1 if enable else 0), "treepo_set_profiling")

    def profile_read(self, kind: int):
        ms, n = ctypes.c_double(), _i64()
        self._check(self.lib.treepo_profile_read(self.h, kind, ctypes.byref(ms), ctypes.byref(n)),
                    "treepo_profile_read")
        return ms.value, n.value


BUDGET_EVEN, BUDGET_HIGH_PROB, BUDGET_LOW_PROB = 0, 1, 2


def branch_budget(scores, total: int, mode: int = BUDGET_EVEN, temperature: float = 2.0) -> list[int]:
    """Branches per active path (treepo_branch_budget); scores: last-segment log probabilities."""
    lib = load_library()
    sc = np.ascontiguousarray(np.asarray(scores, dtype=np.float32))
    out = np.zeros(max(len(sc), 1), dtype=np.int32)
    st = lib.treepo_branch_budget(len(sc), sc.ctypes.data_as(ctypes.POINTER(ctypes.c_float)), int(total), int(mode),
                                  float(temperature), _ptr32(out))
    if st != OK:
        raise TreePOError(st, "treepo_branch_budget: " + lib.treepo_strerror(st).decode())
    return [int(x) for x in out[:len(sc)]]


def bench_copy(dst, src, nbytes: int, stream=None):
    lib = load_library()
    st = lib.treepo_bench_copy(_dev(dst), _dev(src), nbytes, _stream(stream))
    if st != OK:
        raise TreePOError(st, "treepo_bench_copy")


def bench_read(src, nbytes: int, sink, stream=None):
    lib = load_library()
    st = lib.treepo_bench_read(_dev(src), nbytes, _dev(sink), _stream(stream))
    if st != OK:
        raise TreePOError(st, "treepo_bench_read")


def bench_overlap(mode: int, waves_per_simd: int, iters: int, sink, cycles, stream=None):
    lib = load_library()
    st = lib.treepo_bench_overlap(mode, waves_per_simd, iters, _dev(sink), _dev(cycles), _stream(stream))
    if st != OK:
        raise TreePOError(st, "treepo_bench_overlap")


def bench_stream(src, nbytes: int, sink, mode: int, workgroups: int, stream=None):
    lib = load_library()
    st = lib.treepo_bench_stream(_dev(src), nbytes, _dev(sink), mode, workgroups, _stream(stream))
    if st != OK:
        raise TreePOError(st, "treepo_bench_stream")
