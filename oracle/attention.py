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

    Returns o[r][h] = softmax(q[r,h] . K[h, S_r]^T * scale) V[h, S_r] (float64)."""
    rows, H, Dh = q.shape
    out = np.zeros((rows, H, Dh), dtype=np.float64)
    for r in range(rows):
        s_idx = np.asarray(sorted(key_slots[r]), dtype=np.int64)
        K = k_cache[:, s_idx, :]                             # [H][|S|][Dh]
        V = v_cache[:, s_idx, :]
        s = np.einsum("hd,hkd->hk", q[r], K) * scale         # [H][|S|]
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p /= p.sum(axis=1, keepdims=True)
        out[r] = np.einsum("hk,hkd->hd", p, V)
    return out


def tree_key_slots(L: int, anc_self: Sequence[Sequence[int]]):
    """Key slots of each tree row when node j's K/V sit in cache slot L + j:
    [0, L) plus L + j for every j on the node's root-to-node path."""
    base = list(range(L))
    return [base + [L + j for j in a] for a in anc_self]
