"""EAGLE-2 dynamic draft-tree expansion and top-N rerank (Sec. 3.1; Sec. 4.2, Eq. 3-5).

The root's top-k children form layer 1.  Each later layer is produced by one draft
forward over the k frontier nodes; every frontier node proposes its top-k tokens, each
child is scored by the product of confidences along its path (Eq. 3; kept here as the
sum of log-probabilities, which orders identically), all children join the candidate
pool, and the k best children of the layer become the next frontier.  The pool then
has k + (d - 1) k^2 nodes (Eq. 5), and the N best nodes of the pool form the tree that
is verified.

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


def build_tree(root_token: int, pool: Sequence[PoolNode], selected: Sequence[int]) -> Tree:
    """BFS-ordered tree arrays of the selected pool nodes, the root at index 0."""
    order = sorted(selected, key=lambda c: (pool[c].depth, -pool[c].score, pool[c].creation))
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
