"""Pins of the prefill oracle (causal attention of appended tokens over
their chain) against what the mathematics fixes, and planted mistakes that
the pins must catch."""

from __future__ import annotations

import inspect

import numpy as np
import pytest
from scipy.special import logsumexp, softmax

from oracle import attention as A
from oracle import metadata as M
from oracle import prefill as P
from workloads import node_kv_bits, query_bits

SEED = 4242


def _setup(hq=6, hkv=2, d=16, n_root=37, n_child=21):
    """A root prompt of n_root tokens and a child segment of n_child tokens,
    each appended (and prefilled) in its own call."""
    m = M.TreeModel(8, 1000, 100)
    r = m.new_root(n_root)
    m.append([r], [n_root])
    c, = m.fork(r, 1, n_child)
    m.append([c], [n_child])
    kv = {n: node_kv_bits(SEED, n, ln, hkv, d) for n, ln in ((r, n_root), (c, n_child))}
    q = query_bits(SEED, 0, n_root + n_child, hq, d)
    return m, (lambda n: kv[n]), r, c, q


def _f(bits):
    return A.bf16_bits_to_f64(bits)


def _causal_matrix(K, V, Q, scale, prefix):
    """Textbook causal attention in matrix form: S = scale Q K^T with the
    columns past each row's own position set to -inf (row i sits at chain
    position prefix + i); W = row softmax of S; O = W V."""
    hq, hkv = Q.shape[1], K.shape[1]
    n, L = Q.shape[0], K.shape[0]
    out = np.empty((n, hq, V.shape[2]))
    lse = np.empty((n, hq))
    mask = np.arange(L)[None, :] > (prefix + np.arange(n))[:, None]
    for h in range(hq):
        g = h * hkv // hq
        S = scale * Q[:, h, :] @ K[:, g, :].T
        S[mask] = -np.inf
        out[:, h, :] = softmax(S, axis=1) @ V[:, g, :]
        lse[:, h] = logsumexp(S, axis=1)
    return out, lse


def test_first_token_closed_form():
    """The first prompt token sees only itself: out = its V row, lse = its score."""
    m, kv, r, c, q = _setup()
    o, l = P.prefill(m, kv, [r], [37], q[:37], 0.25)
    K, V = _f(kv(r)[0]), _f(kv(r)[1])
    for h in range(6):
        assert np.array_equal(o[0, h], V[0, h // 3])
        assert l[0, h] == pytest.approx(0.25 * float(_f(q[0, h]) @ K[0, h // 3]), abs=1e-12)
    # the second token: two-term softmax written out
    s0 = 0.25 * _f(q[1, 4]) @ K[0, 1]
    s1 = 0.25 * _f(q[1, 4]) @ K[1, 1]
    want = (np.exp(s0) * V[0, 1] + np.exp(s1) * V[1, 1]) / (np.exp(s0) + np.exp(s1))
    assert np.allclose(o[1, 4], want, atol=1e-13, rtol=0)


def test_matches_masked_matrix_form_root_and_child():
    m, kv, r, c, q = _setup()
    o, l = P.prefill(m, kv, [r], [37], q[:37], 0.3)
    K, V = _f(kv(r)[0]), _f(kv(r)[1])
    wo, wl = _causal_matrix(K, V, _f(q[:37]), 0.3, 0)
    assert np.abs(o - wo).max() < 1e-12 and np.abs(l - wl).max() < 1e-12
    # the child segment attends to the whole prompt plus its own earlier tokens
    o, l = P.prefill(m, kv, [c], [21], q[37:], 0.3)
    Kc = np.concatenate([K, _f(kv(c)[0])])
    Vc = np.concatenate([V, _f(kv(c)[1])])
    wo, wl = _causal_matrix(Kc, Vc, _f(q[37:]), 0.3, 37)
    assert np.abs(o - wo).max() < 1e-12 and np.abs(l - wl).max() < 1e-12


def test_last_token_is_the_decode_of_the_chain():
    """The last appended token attends to the whole chain: the decode result."""
    m, kv, r, c, q = _setup()
    o, l = P.prefill(m, kv, [r, c], [37, 21], q, 0.2)
    for x, row in ((r, 36), (c, 57)):
        do, dl = A.tree_decode(m, kv, [x], q[row:row + 1], 0.2)
        assert np.abs(o[row] - do[0]).max() < 1e-13 and np.abs(l[row] - dl[0]).max() < 1e-13


def test_rows_selection_and_empty():
    m, kv, r, c, q = _setup()
    o, l = P.prefill(m, kv, [r, c], [37, 21], q, 0.2)
    so, sl = P.prefill(m, kv, [r, c], [37, 21], q, 0.2, rows=[57, 0, 40])
    assert np.array_equal(so, o[[57, 0, 40]]) and np.array_equal(sl, l[[57, 0, 40]])
    eo, el = P.prefill(m, kv, [r], [0], q[:0], 0.2)
    assert eo.shape == (0, 6, 16) and el.shape == (0, 6)


def _mutant(kind):
    src = inspect.getsource(P.prefill)
    if kind == "exclude_self":
        src = src.replace("K[:p + 1], V[:p + 1]", "K[:max(p, 1)], V[:max(p, 1)]")
    elif kind == "see_next":
        src = src.replace("K[:p + 1], V[:p + 1]", "K[:p + 2], V[:p + 2]")
    elif kind == "no_prefix":
        src = src.replace("first = K.shape[0] - n", "K, V = K[-n:], V[-n:]\n            first = 0")
    elif kind == "positions_from_zero":
        src = src.replace("first = K.shape[0] - n", "first = 0")
    ns = dict(P.__dict__)
    exec(compile(src, "<mutant>", "exec"), ns)
    return ns["prefill"]


@pytest.mark.parametrize("kind", ["exclude_self", "see_next", "no_prefix", "positions_from_zero"])
def test_prefill_mutation_caught(kind, monkeypatch):
    mut = _mutant(kind)
    assert mut is not P.prefill
    monkeypatch.setattr(P, "prefill", mut)
    failed = 0
    for t in (test_first_token_closed_form, test_matches_masked_matrix_form_root_and_child,
              test_last_token_is_the_decode_of_the_chain):
        try:
            t()
        except (AssertionError, ValueError, IndexError):
            failed += 1
    assert failed >= 1


def test_chunking_does_not_change_the_result():
    """Prefilling a prompt in two calls gives the rows of one call: causal
    attention of a token depends only on the chain up to it."""
    hq, hkv, d = 4, 2, 16
    kv_bits = node_kv_bits(SEED + 1, 0, 90, hkv, d)
    q = query_bits(SEED + 1, 0, 90, hq, d)
    one = M.TreeModel(8, 100, 10)
    r = one.new_root(90)
    one.append([r], [90])
    o1, l1 = P.prefill(one, lambda n: kv_bits, [r], [90], q, 0.3)
    two = M.TreeModel(8, 100, 10)
    r2 = two.new_root(90)
    two.append([r2], [55])
    kv55 = (kv_bits[0][:55], kv_bits[1][:55])
    oa, la = P.prefill(two, lambda n: kv55, [r2], [55], q[:55], 0.3)
    two.append([r2], [35])
    ob, lb = P.prefill(two, lambda n: kv_bits, [r2], [35], q[55:], 0.3)
    assert np.array_equal(np.concatenate([oa, ob]), o1) and np.array_equal(np.concatenate([la, lb]), l1)
