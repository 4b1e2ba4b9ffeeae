"""Oracle: hardware-friendly tree building and tree verification. Test infrastructure only.

Sec. 4 ("Hardware friendly tree building process", and its table of how often the second and
third most likely tokens are accepted): instead of one greedy chain, the sparse model drafts a
tree whose every step keeps a fixed number W of leaves (the treewidth). Each leaf is a path
from the root, ranked
by the cumulative log-likelihood of the path under the sparse model; a step expands every
leaf and keeps the W expansions of largest cumulative log-likelihood, like beam search, so
the tree has a fixed shape and only the parent links between steps vary. The full model then
checks the whole tree in one parallel pass, and of the W complete paths the one that
advances furthest is kept.

Readings adopted (the paper gives the procedure in prose and a figure, no formulas):

  * log-likelihoods are log softmax(logits / temperature) of the sparse model at the leaf;
  * a step ranks every (parent leaf, token) pair by parent cumulative log-likelihood plus the
    token's log-likelihood and keeps the W largest; ties go to the lower parent slot, then the
    lower token id; the new leaves are stored best first (slot 0 has the largest value);
  * the first step expands the root, a single distribution with cumulative value 0;
  * verification: node (i, w) carries token x[i][w] and the full model's logits L[i][w] for
    that position (computed on the node's parent path and aligned by the caller);
    q = softmax(L / temperature)[x], 0 for an id outside the vocabulary; a path's advance
    length is its first position with q < r (strict), else K; the kept path has the largest
    advance length, ties to the lower leaf slot; the corrected token is the argmax of the raw
    L at the kept path's rejected node (lowest index on ties), or of the leaf's bonus row when
    all K positions are accepted and bonus rows are given, else -1.

With W = 1 a step keeps the single most likely token and verification is the chain check of
oracle.verify.verify_accept; the tests pin both reductions.
"""

from __future__ import annotations

import numpy as np

from .verify import softmax_row_stats


def log_softmax(logits, temperature: float = 1.0) -> np.ndarray:
    """log softmax(logits / temperature) over the last axis, float64."""
    z = np.asarray(logits, dtype=np.float64) / float(temperature)
    m = np.max(z, axis=-1, keepdims=True)
    return z - m - np.log(np.sum(np.exp(z - m), axis=-1, keepdims=True))


def tree_build_step(logits, cum_ll, width: int, temperature: float = 1.0):
    """One pruned expansion step for one tree.

    logits [Wc, V]: the sparse model's logits at the Wc current leaves (Wc = 1 at the root);
    cum_ll [Wc] or None (the root: 0).
    Returns (tokens [W] int64, parents [W] int64, cum_ll [W] float64), best first.
    """
    ls = log_softmax(np.atleast_2d(logits), temperature)
    wc, v = ls.shape
    base = np.zeros(wc) if cum_ll is None else np.asarray(cum_ll, dtype=np.float64)
    score = (base[:, None] + ls).ravel()
    parent = np.repeat(np.arange(wc), v)
    token = np.tile(np.arange(v), wc)
    order = np.lexsort((token, parent, -score))[:width]  # primary key: larger score first
    return token[order], parent[order], score[order]


def tree_paths(parents) -> np.ndarray:
    """Slot of every step's node on the path to each leaf: [W, K] (parents [K, W])."""
    p = np.asarray(parents)
    k_n, w_n = p.shape
    path = np.zeros((w_n, k_n), dtype=np.int64)
    for leaf in range(w_n):
        w = leaf
        for i in range(k_n - 1, -1, -1):
            path[leaf, i] = w
            if i > 0:
                w = int(p[i, w])
    return path


def tree_verify(logits, tokens, parents, r: float, temperature: float = 1.0, bonus=None):
    """Verification of one tree.

    logits [K, W, V], tokens [K, W], parents [K, W] (row 0 unused), bonus [W, V] or None.
    Returns (best_leaf, accept_len, next_token, q [K, W] float64, advance [W] int64).
    """
    lg = np.asarray(logits)
    tk = np.asarray(tokens)
    k_n, w_n, v_n = lg.shape
    if bonus is not None and np.shape(bonus) != (w_n, v_n):
        raise ValueError("bonus rows must be [W, V], over the same vocabulary as the nodes")
    q = np.zeros((k_n, w_n), dtype=np.float64)
    amax = np.zeros((k_n, w_n), dtype=np.int64)
    for i in range(k_n):
        for w in range(w_n):
            m, s, am = softmax_row_stats(lg[i, w], temperature)
            amax[i, w] = am
            t = int(tk[i, w])
            if 0 <= t < v_n:
                q[i, w] = np.exp(float(lg[i, w, t]) / float(temperature) - m) / s
    path = tree_paths(parents)
    advance = np.full(w_n, k_n, dtype=np.int64)
    for leaf in range(w_n):
        for i in range(k_n):
            if q[i, path[leaf, i]] < r:
                advance[leaf] = i
                break
    best = int(np.argmax(advance))  # first (lowest) slot among the longest advances
    acc = int(advance[best])
    if acc < k_n:
        nxt = int(amax[acc, path[best, acc]])
    elif bonus is not None:
        nxt = int(np.argmax(np.asarray(bonus)[best]))
    else:
        nxt = -1
    return best, acc, nxt, q, advance
