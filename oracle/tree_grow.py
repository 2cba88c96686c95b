"""Float64 reference for level-wise draft-tree growth (test infrastructure).

Sec. 3.5 runs tree drafting with the shape (8, 10, 60): depth 8, top-k 10 at
each level, at most 60 candidate tokens; Sec. 3.1 names the pipeline.  The paper
gives no more than the shape, so the rule below is a reading (t-a), the usual
level-wise best-first growth:

  * level 0's frontier is the root (the last verified token, not a draft node)
    with score 0;
  * at each level every frontier node f turns its drafter logits z_f over the
    vocabulary into log-probabilities lp_f(v) = z_f(v) - logsumexp(z_f) and
    proposes its top-k tokens by logit (ties: the smaller token id first);
  * a proposed child (f, v) scores score(f) + lp_f(v); the next frontier is the
    k best children of the whole level (ties: the smaller frontier index, then
    the better proposal rank);
  * after `depth` levels the tree is the n best of all frontier nodes (ties: the
    shallower node, then the earlier one in its level).  Scores never increase
    along a path (lp <= 0), so the set contains every selected node's parent.
  * Output order: by depth, then by rank within the level; parents index this
    order, -1 for children of the root.

Pins (tests/test_oracle_tree_grow_pins.py): top-k against a plain scan of tiny
vocabularies; log-probabilities exponentiate and sum to 1; k = 1 gives the
greedy chain; a hand-derived two-token example; a full tree (n = depth k)
keeps every frontier node; one level against a brute force over every
(frontier node, vocabulary token) pair; ancestor closure, topological order
and the n best on random cases.
"""
from __future__ import annotations

from typing import List, Tuple

import numpy as np


def log_softmax_topk(logits: np.ndarray, k: int) -> Tuple[np.ndarray, np.ndarray]:
    """Per row: the k largest logits' token ids (descending; ties by smaller id) and their log-probabilities."""
    z = np.asarray(logits, dtype=np.float64)
    m = z.max(axis=-1, keepdims=True)
    lse = m[..., 0] + np.log(np.exp(z - m).sum(axis=-1))
    # stable sort of (-z) keeps the smaller id first among equal logits
    order = np.argsort(-z, axis=-1, kind="stable")[..., :k]
    lp = np.take_along_axis(z, order, axis=-1) - lse[..., None]
    return order.astype(np.int32), lp


def grow_level(scores: np.ndarray, tokens: np.ndarray, logprobs: np.ndarray, k: int):
    """One level for one sequence: frontier scores [F], proposals tokens/logprobs [F][k'].

    Returns (parent index in the frontier, token, score) of the k best children."""
    F, kp = tokens.shape
    cand = []
    for f in range(F):
        for r in range(kp):
            cand.append((-(float(scores[f]) + float(logprobs[f, r])), f, r))
    cand.sort()                       # best score first; ties: smaller frontier index, then better rank
    sel = cand[:k]
    return (np.array([c[1] for c in sel], np.int32), np.array([tokens[c[1], c[2]] for c in sel], np.int32),
            np.array([-c[0] for c in sel], np.float64))


def finalize(levels: List[Tuple[np.ndarray, np.ndarray, np.ndarray]], n: int):
    """The n best nodes of all levels as a tree: (parents, tokens, depths, scores) in output order.

    levels[d] = (parent index in level d - 1's frontier (unused for d = 0), token, score) of level d + 1's
    frontier, in rank order."""
    cand = []
    for d, (_, _, sc) in enumerate(levels):
        for i in range(len(sc)):
            cand.append((-float(sc[i]), d, i))
    cand.sort()                       # ties: shallower, then earlier in its level
    chosen = sorted((d, i) for _, d, i in cand[:n])
    index = {key: j for j, key in enumerate(chosen)}
    parents, toks, depths, scores = [], [], [], []
    for d, i in chosen:
        par, tok, sc = levels[d]
        parents.append(-1 if d == 0 else index[(d - 1, int(par[i]))])
        toks.append(int(tok[i]))
        depths.append(d)
        scores.append(float(sc[i]))
    return (np.array(parents, np.int32), np.array(toks, np.int32), np.array(depths, np.int32),
            np.array(scores, np.float64))


def grow_tree(level_logits: List[np.ndarray], k: int, n: int):
    """Whole growth for one sequence: level_logits[d] is [F_d][V] (F_0 = 1, then k)."""
    scores = np.zeros(1)
    levels = []
    for z in level_logits:
        tok, lp = log_softmax_topk(z, k)
        par, t, sc = grow_level(scores, tok, lp, k)
        levels.append((par, t, sc))
        scores = sc
    return finalize(levels, n)
