"""Plant plausible mistakes in the oracle (on the CPU) and check a pin catches each.

A pin set that passes a wrong oracle proves nothing; each mutation below is a
mistake one could make writing the definition (a wrong KV-head map, a dropped
scale, a dropped root segment, swapped operands, a wrong start offset, a
missing LSE weight) and must make at least one pin fail.
"""

import numpy as np
import pytest

from oracle import attention as A
from oracle import cascade as C
from oracle import metadata as M
from tests import oracle_pins as P


def _attend_factory(kind):
    def attend(q, K, V, scale):
        hq, hkv = q.shape[0], K.shape[1]
        group = hq // hkv
        out = np.empty((hq, V.shape[2]))
        lse = np.empty(hq)
        for h in range(hq):
            g = (h % hkv) if kind == "interleaved_heads" else h // group
            sc = 1.0 if kind == "no_scale" else scale
            s = sc * (K[:, g, :] @ q[h])
            m = s.max()
            e = np.exp(s - m)
            z = e.sum()
            vals = K if kind == "k_as_v" else V
            out[h] = (e @ vals[:, g, :]) / (len(e) if kind == "mean_norm" else z)
            lse[h] = (np.log(z) if kind == "lse_no_max" else m + np.log(z))
        return out, lse
    return attend


def _materialize_drop_root(model, node_kv, x, cache=None):
    ks, vs = [], []
    for n in model.chain(x)[1:] or model.chain(x):
        ln = model.nodes[n]["len"]
        kb, vb = node_kv(n)
        ks.append(A.bf16_bits_to_f64(kb[:ln])); vs.append(A.bf16_bits_to_f64(vb[:ln]))
    return np.concatenate(ks), np.concatenate(vs)


def _materialize_off_by_one(model, node_kv, x, cache=None):
    ks, vs = [], []
    for n in model.chain(x):
        ln = model.nodes[n]["len"]
        kb, vb = node_kv(n)
        lo = 1 if ln > 1 else 0
        ks.append(A.bf16_bits_to_f64(kb[lo:ln])); vs.append(A.bf16_bits_to_f64(vb[lo:ln]))
    return np.concatenate(ks), np.concatenate(vs)


def _make_factory(kind):
    orig = M.TreeModel._make

    def _make(self, parent, depth, start, cap, tree_id):
        if kind == "start_ignores_len" and parent >= 0:
            start = self.nodes[parent]["start"]
        if kind == "depth_not_incremented" and parent >= 0:
            depth = self.nodes[parent]["depth"]
        nid = orig(self, parent, depth, start, cap, tree_id)
        if kind == "blocks_off_by_one" and nid > 0:
            self.nodes[nid]["block_begin"] += 1
        return nid
    return _make


def _combine_factory(kind):
    def combine(parts):
        ms = np.array([p[1] for p in parts])
        m_star = ms.max()
        w = np.exp(ms - m_star)
        if kind == "unweighted_l":
            L = sum(p[2] for p in parts)
        else:
            L = sum(wi * p[2] for wi, p in zip(w, parts))
        if kind == "unweighted_o":
            O = sum(p[0] for p in parts)
        else:
            O = sum(wi * p[0] for wi, p in zip(w, parts))
        return O / L, m_star + np.log(L)
    return combine


def _widen_factory(kind):
    def widen(bits):
        b = np.asarray(bits, dtype=np.uint16)
        if kind == "shift_without_widening":
            # the shift done in 16 bits: every value becomes 0
            return (b << np.uint16(8) << np.uint16(8)).astype(np.float64)
        if kind == "sign_dropped":
            u = (b & np.uint16(0x7FFF)).astype(np.uint32) << np.uint32(16)
        else:  # "fraction_truncated": the low fraction bits lost
            u = (b & np.uint16(0xFFF0)).astype(np.uint32) << np.uint32(16)
        return u.view(np.float32).astype(np.float64)
    return widen


_orig_tree_decode = A.tree_decode


def _decode_positions_sorted(model, node_kv, leaves, q_bits, scale, positions=None):
    return _orig_tree_decode(model, node_kv, leaves, q_bits, scale,
                             positions=None if positions is None else sorted(positions))


MUTATIONS = {
    "shift_without_widening": (A, "bf16_bits_to_f64", _widen_factory("shift_without_widening")),
    "sign_dropped": (A, "bf16_bits_to_f64", _widen_factory("sign_dropped")),
    "fraction_truncated": (A, "bf16_bits_to_f64", _widen_factory("fraction_truncated")),
    "positions_sorted": (A, "tree_decode", _decode_positions_sorted),
    "interleaved_heads": (A, "attend", _attend_factory("interleaved_heads")),
    "no_scale": (A, "attend", _attend_factory("no_scale")),
    "k_as_v": (A, "attend", _attend_factory("k_as_v")),
    "mean_norm": (A, "attend", _attend_factory("mean_norm")),
    "lse_no_max": (A, "attend", _attend_factory("lse_no_max")),
    "drop_root": (A, "materialize", _materialize_drop_root),
    "skip_first_row": (A, "materialize", _materialize_off_by_one),
    "start_ignores_len": (M.TreeModel, "_make", _make_factory("start_ignores_len")),
    "depth_not_incremented": (M.TreeModel, "_make", _make_factory("depth_not_incremented")),
    "blocks_off_by_one": (M.TreeModel, "_make", _make_factory("blocks_off_by_one")),
    "unweighted_l": (C, "combine", _combine_factory("unweighted_l")),
    "unweighted_o": (C, "combine", _combine_factory("unweighted_o")),
}

FAST_PINS = [p for p in P.ALL_PINS if p is not P.pin_long_context_counts]


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_mutation_is_caught(name, monkeypatch):
    obj, attr, repl = MUTATIONS[name]
    monkeypatch.setattr(obj, attr, repl)
    failed = []
    for pin in FAST_PINS:
        try:
            if pin is P.pin_bruteforce:
                pin(seeds=(1, 2))
            elif pin is P.pin_structure_invariants:
                pin(cfgs=(1, 2, 4))
            else:
                pin()
        except (AssertionError, IndexError, ValueError):
            failed.append(pin.__name__)
    assert failed, f"mutation {name} passed every pin"


# ---- the TreePO advantage oracle ----------------------------------------------

from oracle import advantage as ADV  # noqa: E402
from tests import advantage_pins as AP  # noqa: E402


def _adv_factory(kind):
    def subgroups(parents, leaves, rewards):
        chains = [ADV.chain(parents, int(x)) for x in leaves]
        members = {}
        for p, ch in enumerate(chains):
            for a in ch:
                members.setdefault(a, []).append(p)
        R = np.asarray(rewards, dtype=np.float64)
        rows = []
        for p, ch in enumerate(chains):
            preds = ch if kind == "own_node_group" else ch[:-1]
            row = []
            for a in preds:
                g = members[a]
                if kind == "leave_one_out":
                    others = [k for k in g if k != p] or g
                    base = R[others].mean()
                else:
                    base = R[g].mean()
                row.append((a, len(g), R[p] - base))
            rows.append(row)
        return rows, chains

    def tree_advantage(parents, leaves, rewards, weighting="mean"):
        R = np.asarray(rewards, dtype=np.float64)
        n = len(leaves)
        rows, chains = subgroups(parents, leaves, rewards)
        roots = [ch[0] for ch in chains]
        kept = []
        for p in range(n):
            g = [k for k in range(n) if roots[k] == roots[p]]
            kept.append(kind == "no_rejection" or bool(np.std(R[g]) != 0.0))
        adv = np.zeros(n)
        pooled = np.zeros(n)
        for p in range(n):
            if not rows[p]:
                continue
            a = np.array([x for (_, _, x) in rows[p]])
            w = np.array([s for (_, s, _) in rows[p]], dtype=float)
            if kind == "inverse_size":
                w = 1.0 / w
            pooled[p] = a.mean() if weighting == "mean" else (w * a).sum() / w.sum()
        pairs = [x for p in range(n) if kept[p] for (_, _, x) in rows[p]]
        if not pairs:
            return adv
        if kind == "ddof1":
            sigma = float(np.std(pairs, ddof=1))
        elif kind == "pooled_std":
            sigma = float(np.std([pooled[p] for p in range(n) if kept[p] and rows[p]]))
        else:
            sigma = float(np.std(pairs))
        for p in range(n):
            if kept[p] and rows[p]:
                s = sigma
                if kind == "per_query_std":
                    s = float(np.std([x for k in range(n) if roots[k] == roots[p] for (_, _, x) in rows[k]]))
                adv[p] = pooled[p] / s if s > 0 else 0.0
        return adv

    return subgroups, tree_advantage


@pytest.mark.parametrize("kind", ["own_node_group", "leave_one_out", "no_rejection", "inverse_size", "ddof1",
                                  "pooled_std", "per_query_std"])
def test_advantage_mutation_caught(kind, monkeypatch):
    subgroups, adv = _adv_factory(kind)
    monkeypatch.setattr(ADV, "subgroup_advantages", subgroups)
    monkeypatch.setattr(ADV, "tree_advantage", adv)
    failed = []
    for pin in AP.ALL:
        try:
            pin()
        except AssertionError:
            failed.append(pin.__name__)
    assert failed, f"mutation {kind} passed every advantage pin"


def test_advantage_mutation_factory_faithful():
    """The unmutated copy used above reproduces the oracle (so a caught
    mutation is caught for its planted mistake)."""
    _, adv = _adv_factory("none")
    parents, leaves = AP.random_forest(5)
    R = np.random.default_rng(5).normal(size=len(leaves))
    for w in ("mean", "size"):
        assert np.abs(adv(parents, leaves, R, w) - ADV.tree_advantage(parents, leaves, R, w)).max() <= 1e-12


# ---- the branching-budget oracle ----------------------------------------------

import math  # noqa: E402

from oracle import budget as BUD  # noqa: E402
from tests import test_oracle_budget as BP  # noqa: E402


def _budget_factory(kind):
    orig_weights = BUD.weights

    def branch_budget(scores, total, mode="even", temperature=2.0):
        n = len(scores)
        t = 1.0 if kind == "no_temperature" and mode != "even" else temperature
        w = orig_weights(scores, mode, t)
        rest = total if kind == "no_min_one" else max(total - n, 0)
        quota = [rest * x for x in w]
        base = [int(math.floor(q)) for q in quota]
        left = rest - sum(base)
        if kind == "ties_high_index":
            order = sorted(range(n), key=lambda k: (-(quota[k] - base[k]), -k))
        else:
            order = sorted(range(n), key=lambda k: (-(quota[k] - base[k]), k))
        if kind != "drop_remainder":
            for k in order[:left]:
                base[k] += 1
        return base if kind == "no_min_one" else [1 + b for b in base]
    return branch_budget


@pytest.mark.parametrize("kind", ["no_temperature", "no_min_one", "ties_high_index", "drop_remainder"])
def test_budget_mutation_caught(kind, monkeypatch):
    monkeypatch.setattr(BUD, "branch_budget", _budget_factory(kind))
    pins = [BP.test_even_transfer_closed_form, lambda: BP.test_sum_min_one_and_order("high"),
            lambda: BP.test_sum_min_one_and_order("low"), BP.test_two_paths_closed_form,
            BP.test_largest_remainder_ties_to_lower_index]
    failed = 0
    for pin in pins:
        try:
            pin()
        except AssertionError:
            failed += 1
    assert failed, f"budget mutation {kind} passed every pin"
