"""Pins of the oracle's verifier-side steps (CPU): the additive attention bias
of the draft block (tree attention, Preliminaries) and the commit of the
accepted path's key/value rows.

The bias is checked against ancestor sets rebuilt by walking the parent
indices (independent of the bitset mask) and against the attention it
induces; the row commit against numpy's take on the same rows."""
import numpy as np
import pytest

import oracle

from test_oracle_pins import _random_case, _staged  # noqa: E402


def _ancestor_sets(parents, n):
    out = []
    for i in range(n):
        s, j = {i}, parents[i]
        while j >= 0:
            s.add(int(j))
            j = parents[j]
        out.append(s)
    return out


@pytest.mark.parametrize("seed", range(6))
def test_bias_is_ancestor_closure(seed):
    g = np.random.default_rng(700 + seed)
    L, K = int(g.integers(1, 5)), int(g.integers(1, 4))
    cand, edge = _random_case(g, L, K)
    n_max = 64 if seed % 2 else 70          # 70: two mask words, a ragged one
    budget = int(g.integers(0, n_max + 1))
    r = _staged(L, K, n_max, cand, edge, budget)
    n = r["n_nodes"]
    bias = oracle.mask_to_bias(n, r["mask"])
    anc = _ancestor_sets(r["parents"], n)
    for i in range(n_max):
        for j in range(n_max):
            want = 0.0 if (i < n and j < n and j in anc[i]) else -np.inf
            assert bias[i, j] == want, (i, j)
    # row i sees exactly depth(i) nodes: itself and its ancestors
    assert [(bias[i] == 0).sum() for i in range(n)] == [len(a) for a in anc]


def test_bias_attention_weights_vanish_outside_the_path():
    """softmax(scores + bias) puts weight only on a node's ancestors and
    itself; on them it is the plain softmax of those scores."""
    r = _staged(3, 2, 8, np.array([[20, 10], [5, 30], [7, 3]], np.int32),
                np.array([[[-1, -2], [0, 0]], [[-0.5, -3], [-0.25, -0.75]],
                          [[-0.5, -4], [-1, -0.125]]], np.float32), 6)
    n = r["n_nodes"]
    bias = oracle.mask_to_bias(n, r["mask"])[:n, :n]
    g = np.random.default_rng(5)
    s = g.standard_normal((n, n))
    z = s + bias
    w = np.exp(z - z.max(1, keepdims=True))
    w /= w.sum(1, keepdims=True)
    anc = _ancestor_sets(r["parents"], n)
    for i in range(n):
        idx = sorted(anc[i])
        ref = np.exp(s[i, idx] - s[i, idx].max())
        ref /= ref.sum()
        assert np.allclose(w[i, idx], ref, rtol=1e-14, atol=0)
        assert all(w[i, j] == 0.0 for j in range(n) if j not in anc[i])


@pytest.mark.parametrize("seed", range(5))
def test_gather_rows_is_take(seed):
    g = np.random.default_rng(800 + seed)
    n, row = int(g.integers(1, 40)), int(g.integers(1, 9)) * 16
    src = g.integers(0, 256, size=(n, row), dtype=np.uint8)
    a = int(g.integers(0, min(n, 12) + 1))
    nodes = np.sort(g.choice(n, size=a, replace=False)).astype(np.int32)
    dst = g.integers(0, 256, size=(n, row), dtype=np.uint8)
    before = dst.copy()
    oracle.gather_rows(a, nodes, src, dst)
    assert np.array_equal(dst[:a], np.take(src, nodes, axis=0))
    assert np.array_equal(dst[a:], before[a:])
    # in place: the same result as out of place, rows past acc_len untouched
    inplace = src.copy()
    oracle.gather_rows(a, nodes, inplace, inplace)
    assert np.array_equal(inplace[:a], np.take(src, nodes, axis=0))
    assert np.array_equal(inplace[a:], src[a:])


def test_commit_after_acceptance_keeps_the_accepted_tokens():
    """Acceptance then the row commit: with row i of the block holding node i's
    token, the committed rows spell the accepted tokens in path order."""
    tokens = np.array([7, 9, 3, 5, 8, 2], np.int32)
    parents = np.array([-1, -1, 0, 0, 1, 3], np.int32)
    a, nodes, bonus = oracle.accept(6, tokens, parents, 4,
                                    target_depth=np.array([7, 5, 2, 6, 0], np.int32))
    kv = np.zeros((6, 16), np.int32)
    kv[:, 0] = tokens
    oracle.gather_rows(a, nodes[:a], kv.view(np.uint8), kv.view(np.uint8))
    assert kv[:a, 0].tolist() == [7, 5, 2] and bonus == 6
