"""Pins for the level-wise tree-growth oracle (Sec. 3.5, tree shape (8, 10, 60);
the selection rule is a reading, see oracle/tree_grow.py).

- top-k and log-softmax against a pure-Python scan (ties by smaller token id);
- log-probabilities of the whole vocabulary exponentiate and sum to one;
- k = 1 grows the greedy chain;
- a hand-derived example on a two-token vocabulary (every score is a sum of
  log 0.9 and log 0.1, so the order of the nodes is known in closed form);
- on random cases: n nodes, parents before children, every parent selected,
  scores never increasing along a path, and the kept set being the n best.
"""
import math

import numpy as np
import pytest

from oracle.tree_grow import finalize, grow_level, grow_tree, log_softmax_topk


def scan_topk(row, k):
    best = []
    for v, z in enumerate(row):
        best.append((-z, v))
    best.sort()
    lse = math.log(math.fsum(math.exp(z) for z in row))
    return [v for _, v in best[:k]], [-nz - lse for nz, _ in best[:k]]


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_topk_and_logprobs_match_a_plain_scan(seed):
    rng = np.random.default_rng(seed)
    z = np.round(rng.standard_normal((5, 40)) * 2, 1)          # rounded: many equal logits
    tok, lp = log_softmax_topk(z, 7)
    for r in range(5):
        st, sl = scan_topk(list(z[r]), 7)
        assert tok[r].tolist() == st
        np.testing.assert_allclose(lp[r], sl, rtol=0, atol=1e-12)


def test_full_vocabulary_logprobs_sum_to_one():
    z = np.random.default_rng(3).standard_normal((3, 50)) * 5
    _, lp = log_softmax_topk(z, 50)
    np.testing.assert_allclose(np.exp(lp).sum(axis=1), 1.0, rtol=0, atol=1e-12)


def test_k1_grows_the_greedy_chain():
    rng = np.random.default_rng(4)
    levels = [rng.standard_normal((1, 30)) for _ in range(5)]
    parents, tokens, depths, scores = grow_tree(levels, 1, 5)
    assert parents.tolist() == [-1, 0, 1, 2, 3]
    assert tokens.tolist() == [int(np.argmax(z[0])) for z in levels]
    assert depths.tolist() == [0, 1, 2, 3, 4]


def test_two_token_vocabulary_example():
    # every frontier node proposes token 0 with p = 0.9 and token 1 with p = 0.1 (k = 2, depth 3).
    # A path's score is a log 0.9 + b log 0.1 with a + b = depth; order by the number of 1s, ties
    # by frontier rank, then proposal rank:
    #   level 1: [0] (0 ones), [1] (1 one)
    #   level 2 candidates: 00 (0), 01 (1), 10 (1), 11 (2) -> keep 00, 01 (01 beats 10: its parent ranks first)
    #   level 3 candidates: 000 (0), 001 (1), 010 (1), 011 (2) -> keep 000, 001
    # the 4 best of the 6 frontier nodes: 0 (0), 00 (0), 000 (0) and, among the one-1 nodes 1 (depth 0),
    # 01 (depth 1), 001 (depth 2), the shallowest: 1
    row = np.log(np.array([[0.9, 0.1]]))
    levels = [row, np.repeat(row, 2, axis=0), np.repeat(row, 2, axis=0)]
    parents, tokens, depths, scores = grow_tree(levels, 2, 4)
    assert depths.tolist() == [0, 0, 1, 2]
    assert tokens.tolist() == [0, 1, 0, 0]
    assert parents.tolist() == [-1, -1, 0, 2]
    l9, l1 = math.log(0.9), math.log(0.1)
    np.testing.assert_allclose(scores, [l9, l1, 2 * l9, 3 * l9], rtol=0, atol=1e-12)
    # with all six kept the one-1 nodes follow in depth order
    p6, t6, d6, s6 = grow_tree(levels, 2, 6)
    assert d6.tolist() == [0, 0, 1, 1, 2, 2] and t6.tolist() == [0, 1, 0, 1, 0, 1]
    assert p6.tolist() == [-1, -1, 0, 0, 2, 2]


@pytest.mark.parametrize("seed", range(6))
def test_random_trees_are_closed_ordered_and_best(seed):
    rng = np.random.default_rng(seed)
    depth, k, n, V = 5, 4, 13, 60
    levels = [rng.standard_normal((1 if d == 0 else k, V)) * 3 for d in range(depth)]
    parents, tokens, depths, scores = grow_tree(levels, k, n)
    assert len(parents) == n
    for i in range(n):
        p = parents[i]
        assert (p == -1) == (depths[i] == 0)
        if p >= 0:
            assert p < i and depths[p] == depths[i] - 1 and scores[i] <= scores[p]
    # the kept nodes are the n best of all depth * k frontier nodes
    sc = np.zeros(1)
    every = []
    for z in levels:
        tok, lp = log_softmax_topk(z, k)
        par, t, s = grow_level(sc, tok, lp, k)
        every += list(s)
        sc = s
    assert np.isclose(min(scores), sorted(every, reverse=True)[n - 1], rtol=0, atol=1e-12)


def test_full_tree_keeps_every_frontier_node():
    rng = np.random.default_rng(9)
    levels = [rng.standard_normal((1 if d == 0 else 3, 20)) for d in range(4)]
    parents, tokens, depths, scores = grow_tree(levels, 3, 12)
    assert depths.tolist() == [0] * 3 + [1] * 3 + [2] * 3 + [3] * 3
    assert finalize([(np.zeros(2, np.int32), np.array([5, 6], np.int32), np.array([-1.0, -2.0]))], 1)[1].tolist() == [5]


def brute_force_level(scores, z, k):
    """The k best children over every (frontier node, vocabulary token) pair, with the full log-softmax of
    each row; ties by the smaller frontier index, then the larger logit, then the smaller token id."""
    F, V = z.shape
    cand = []
    for f in range(F):
        lse = math.log(math.fsum(math.exp(x) for x in z[f]))
        for v in range(V):
            cand.append((-(scores[f] + z[f, v] - lse), f, -z[f, v], v))
    cand.sort()
    return [(c[1], c[3], -c[0]) for c in cand[:k]]


@pytest.mark.parametrize("seed", range(8))
def test_level_equals_brute_force_over_the_whole_vocabulary(seed):
    # proposing only each node's top k loses no child of the level's k best (and keeps the tie order)
    rng = np.random.default_rng(100 + seed)
    F, V, k = 4, 9, 3
    z = np.round(rng.standard_normal((F, V)) * 2, 0)             # coarse: ties between and within rows
    scores = np.round(-rng.uniform(0, 3, size=F), 0)
    tok, lp = log_softmax_topk(z, k)
    par, t, sc = grow_level(scores, tok, lp, k)
    want = brute_force_level(scores, z, k)
    assert [(int(a), int(b)) for a, b in zip(par, t)] == [(f, v) for f, v, _ in want]
    np.testing.assert_allclose(sc, [s for _, _, s in want], rtol=0, atol=1e-12)
