"""EAGLE-2 dynamic draft-tree expansion and top-N rerank (Sec. 3.1; Sec. 4.2, Eq. 3-5).

The root's top-k children form layer 1.  Each later layer is produced by one draft
forward over the k frontier nodes; every frontier node proposes its top-k tokens, each
child is scored by the product of confidences along its path (Eq. 3; kept here as the
sum of log-probabilities, which orders identically), all children join the candidate
pool, and the k best children of the layer become the next frontier.  The pool then
has k + (d - 1) k^2 nodes (Eq. 5), and the N best nodes of the pool form the tree that
is verified.

With stochastic children (Sec. 3.1 read literally: children sampled from q) every expanded
node draws its children from q instead of taking its top-k, and no drawn child is dropped;
see expand_sampled.

Readings where the paper is silent:
  * q is the draft softmax at temperature 1 over the allowed ids; log q = logit - lse;
  * ties: top-k by (logit desc, id asc); frontier by (score desc, creation asc); rerank
    by (score desc, depth asc, creation asc); output order is BFS by
    (depth asc, score desc, creation asc), the root at index 0;
  * a node proposes min(k, #allowed ids) children.

Test infrastructure only; see the package docstring.
"""
from __future__ import annotations

import dataclasses
from typing import Callable, List, Sequence, Tuple

import numpy as np

from .numerics import draw_below, uniform_u64_tagged


@dataclasses.dataclass
class PoolNode:
    token: int
    score: float       # sum of log q along the path root..node
    depth: int         # 1 for children of the root
    parent: int        # pool index of the parent, -1 for the root
    creation: int      # pool index (creation order)


@dataclasses.dataclass
class Tree:
    parent: np.ndarray   # [n] int32, -1 for the root (index 0)
    token: np.ndarray    # [n] int32; token[0] is the root token
    depth: np.ndarray    # [n] int32
    score: np.ndarray    # [n] float64; 0 for the root
    pool_index: np.ndarray  # [n] pool index of each draft node (-1 for the root)

    @property
    def n(self) -> int:
        return len(self.parent)


def top_children(logit_row: np.ndarray, lo: int, hi: int, k: int) -> Tuple[np.ndarray, np.ndarray]:
    """Top-k ids of the allowed range [lo, hi) by (logit desc, id asc), with their log q."""
    seg = np.asarray(logit_row[lo:hi], dtype=np.float64)
    mx = seg.max()
    lse = mx + np.log(np.sum(np.exp(seg - mx)))
    ids = np.arange(lo, hi)
    order = np.lexsort((ids, -seg))[: min(k, hi - lo)]
    return ids[order], seg[order] - lse


def expand(root_logits: np.ndarray, level_fn: Callable[[List[int], List[PoolNode]], np.ndarray],
           d_hat: int, k_hat: int, n_budget: int,
           allowed_at_depth: Callable[[int], Tuple[int, int]]) -> Tuple[List[PoolNode], List[int]]:
    """Build the candidate pool.  level_fn(frontier pool indices, pool) returns the draft
    logits of those frontier nodes, one row each.  Returns (pool, selected pool indices)."""
    pool: List[PoolNode] = []

    def add_children(row: np.ndarray, parent: int, parent_score: float, depth: int) -> List[int]:
        lo, hi = allowed_at_depth(depth)
        ids, logq = top_children(row, lo, hi, k_hat)
        made = []
        for t, lq in zip(ids, logq):
            pool.append(PoolNode(int(t), parent_score + float(lq), depth, parent, len(pool)))
            made.append(len(pool) - 1)
        return made

    frontier = add_children(root_logits, -1, 0.0, 1)
    for depth in range(2, d_hat + 1):
        rows = level_fn(frontier, pool)
        made: List[int] = []
        for i, u in enumerate(frontier):
            made += add_children(rows[i], u, pool[u].score, depth)
        made.sort(key=lambda c: (-pool[c].score, pool[c].creation))
        frontier = made[:k_hat]
    ranked = sorted(range(len(pool)), key=lambda c: (-pool[c].score, pool[c].depth, pool[c].creation))
    return pool, ranked[:n_budget]


CHILD_DRAW_TAG = 2


def sampled_children(logit_row: np.ndarray, lo: int, hi: int, n_children: int, temperature: float, top_k: int,
                     seed: int, step: int, parent_node: int) -> Tuple[List[int], List[float]]:
    """Children drawn i.i.d. from q (Sec. 3.1: each selected node generates its children by
    sampling from the draft distribution).  q is the draft softmax at temperature T over the
    allowed ids, truncated to top_k, in the acceptance's integer weights; draw j takes
    r = floor(U W / 2^64) with U from Philox at counter (step, parent_node, j, 2) and returns
    the smallest id whose prefix weight exceeds r.  parent_node is the parent's index in the
    finished tree.  The returned scores are log q at T = 1 over the allowed ids (the
    confidences that rank the frontier)."""
    from .accept import inverse_cdf, quantised_weights
    w = quantised_weights(logit_row, lo, hi, temperature, top_k)
    W = int(sum(int(v) for v in w))
    ids = [inverse_cdf(w, draw_below(uniform_u64_tagged(seed, step, parent_node, j, CHILD_DRAW_TAG), W))
           for j in range(n_children)]
    seg = np.asarray(logit_row[lo:hi], dtype=np.float64)
    mx = seg.max()
    lse = mx + np.log(np.sum(np.exp(seg - mx)))
    return ids, [float(seg[i - lo] - lse) for i in ids]


def expand_sampled(root_logits: np.ndarray, level_fn: Callable[[List[int], List[PoolNode]], np.ndarray],
                   d_hat: int, k_hat: int, n_children: int, n_budget: int,
                   allowed_at_depth: Callable[[int], Tuple[int, int]], *, temperature: float, top_k: int,
                   seed: int, step: int) -> Tuple[List[PoolNode], List[int]]:
    """Stochastic children: every expanded node draws n_children children from q and all of
    them stay in the tree (dropping drawn children by their value would make the siblings
    of a node no longer an i.i.d. sample of q, which the literal Eq. 1 acceptance relies
    on).  Layer 1 is the root's children; each later layer expands the k_hat best nodes of
    the previous layer by path confidence (score desc, creation asc), as many as the budget
    of n_budget draft nodes still admits whole.  Pool order is creation order, depth by
    depth, so a node's tree index is its pool index + 1 and siblings keep their draw order.
    Returns (pool, all pool indices)."""
    assert 1 <= n_children <= n_budget
    pool: List[PoolNode] = []

    def add_children(row: np.ndarray, parent: int, parent_score: float, depth: int) -> List[int]:
        lo, hi = allowed_at_depth(depth)
        ids, logq = sampled_children(row, lo, hi, n_children, temperature, top_k, seed, step, parent + 1)
        made = []
        for t, lq in zip(ids, logq):
            pool.append(PoolNode(int(t), parent_score + lq, depth, parent, len(pool)))
            made.append(len(pool) - 1)
        return made

    layer = add_children(root_logits, -1, 0.0, 1)
    for depth in range(2, d_hat + 1):
        nf = min(k_hat, len(layer), (n_budget - len(pool)) // n_children)
        if nf <= 0:
            break
        frontier = sorted(layer, key=lambda c: (-pool[c].score, pool[c].creation))[:nf]
        rows = level_fn(frontier, pool)
        layer = []
        for i, u in enumerate(frontier):
            layer += add_children(rows[i], u, pool[u].score, depth)
    return pool, list(range(len(pool)))


def build_tree(root_token: int, pool: Sequence[PoolNode], selected: Sequence[int], by_creation: bool = False) -> Tree:
    """BFS-ordered tree arrays of the selected pool nodes, the root at index 0: by (depth,
    score desc, creation), or with by_creation by (depth, creation) (stochastic children,
    whose siblings keep their draw order)."""
    key = (lambda c: (pool[c].depth, pool[c].creation)) if by_creation else \
        (lambda c: (pool[c].depth, -pool[c].score, pool[c].creation))
    order = sorted(selected, key=key)
    index_of = {c: i + 1 for i, c in enumerate(order)}
    n = len(order) + 1
    parent = np.full(n, -1, dtype=np.int32)
    token = np.zeros(n, dtype=np.int32)
    depth = np.zeros(n, dtype=np.int32)
    score = np.zeros(n, dtype=np.float64)
    pidx = np.full(n, -1, dtype=np.int64)
    token[0] = root_token
    for c, i in index_of.items():
        p = pool[c].parent
        parent[i] = 0 if p == -1 else index_of[p]     # selection is closed under ancestors
        token[i] = pool[c].token
        depth[i] = pool[c].depth
        score[i] = pool[c].score
        pidx[i] = c
    return Tree(parent, token, depth, score, pidx)


def pool_size(d_hat: int, k_hat: int) -> int:
    """Eq. 5: k + (d - 1) k^2 candidates when every node proposes k children."""
    return k_hat + (d_hat - 1) * k_hat * k_hat
