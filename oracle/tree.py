"""Ancestor sets of a draft tree (Sec. 3.1: each node's context is the prefix plus the
path from the root to the node, the 'tree mask').

Test infrastructure only; see the package docstring.
"""
from __future__ import annotations

from typing import List, Sequence

import numpy as np


def ancestors_and_self(parent: Sequence[int]) -> List[List[int]]:
    """For each node i, the sorted list of nodes on the path root..i (i included).

    Walks the parent pointers up to the root (parent -1)."""
    out = []
    for i in range(len(parent)):
        path = []
        u = i
        while u != -1:
            path.append(u)
            u = int(parent[u])
        out.append(sorted(path))
    return out


def packed_mask(parent: Sequence[int], words: int) -> np.ndarray:
    """uint64 [n][words]: bit j of row i (word j // 64, bit j % 64) is set iff node j lies
    on the path root..i."""
    n = len(parent)
    m = np.zeros((n, words), dtype=np.uint64)
    for i, anc in enumerate(ancestors_and_self(parent)):
        for j in anc:
            m[i, j // 64] |= np.uint64(1) << np.uint64(j % 64)
    return m


def depths(parent: Sequence[int]) -> np.ndarray:
    return np.array([len(a) - 1 for a in ancestors_and_self(parent)], dtype=np.int32)


def is_bfs_ordered(parent: Sequence[int]) -> bool:
    """Root first, every parent before its child, depths non-decreasing."""
    if len(parent) == 0 or parent[0] != -1:
        return False
    d = depths(parent)
    return all(0 <= parent[i] < i for i in range(1, len(parent))) and bool(np.all(np.diff(d) >= 0))
