"""Tree attention by its definition (Sec. 3.1): node i's query attends to exactly the keys
of the committed prefix and of the nodes on its root-to-node path.

Test infrastructure only; see the package docstring.
"""
from __future__ import annotations

from typing import Sequence

import numpy as np


def attend_rows(q: np.ndarray, k_cache: np.ndarray, v_cache: np.ndarray,
                key_slots: Sequence[Sequence[int]], scale: float) -> np.ndarray:
    """q: [rows][H][Dh]; caches: [H][S][Dh]; key_slots[r]: the cache slots row r may see.

    Returns o[r][h] = softmax(q[r,h] . K[h, S_r]^T * scale) V[h, S_r] (float64).  All rows
    are evaluated together over the union of their key sets, each row's scores outside its
    own set S_r removed (weight exactly 0) before the softmax."""
    rows, H, Dh = q.shape
    used = np.asarray(sorted(set().union(*[set(int(j) for j in ks) for ks in key_slots])), dtype=np.int64)
    col = {int(j): c for c, j in enumerate(used)}
    allowed = np.zeros((rows, len(used)), dtype=bool)
    for r, ks in enumerate(key_slots):
        allowed[r, [col[int(j)] for j in ks]] = True
    K = k_cache[:, used, :]                                  # [H][U][Dh]
    V = v_cache[:, used, :]
    s = np.matmul(q.transpose(1, 0, 2), K.transpose(0, 2, 1)) * scale   # [H][rows][U]
    s = np.where(allowed[None], s, -np.inf)
    s = s - s.max(axis=2, keepdims=True)
    p = np.exp(s)
    p /= p.sum(axis=2, keepdims=True)
    return np.matmul(p, V).transpose(1, 0, 2)                # [rows][H][Dh]


def tree_key_slots(L: int, anc_self: Sequence[Sequence[int]]):
    """Key slots of each tree row when node j's K/V sit in cache slot L + j:
    [0, L) plus L + j for every j on the node's root-to-node path."""
    base = list(range(L))
    return [base + [L + j for j in a] for a in anc_self]
