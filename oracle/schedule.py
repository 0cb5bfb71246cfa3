"""Tree depth and width per cycle (Sec. 4): adjacent initialisation (Sec. 4.1, Horizontal
Repeat) followed by bisectional dynamic adaptation (Sec. 4.2, Eq. 2) and the bounds of
Sec. 4.2.

Readings where the paper is silent:
  * the initial attributes of the tree for cell (i, j) are the (depth, width) of the tree
    whose cycle committed cell (i, j-1); at j = 0 the raster predecessor is used, and the
    first tree (no record yet) takes (d0, k0) without adaptation;
  * the acceptance rate is alpha = a / d, a counting accepted draft tokens only, so with
    beta = 1 a tree is 'positive' iff every drafted layer was accepted;
  * the bounds are inclusive ranges applied after Eq. 2, to depth and width alike;
  * near the end of the image the depth is cut to the tokens that remain minus one
    (the bonus token), and a depth of 0 means a plain AR step.

Test infrastructure only; see the package docstring.
"""
from __future__ import annotations

from typing import Optional, Tuple

from synth import SchedCfg


def clamp(x: int, lo: int, hi: int) -> int:
    return max(lo, min(hi, x))


def bisect(d_init: int, k_init: int, alpha_num: int, alpha_den: int, cfg: SchedCfg) -> Tuple[int, int]:
    """Eq. 2: deeper and narrower when alpha >= beta, shallower and wider otherwise.
    alpha = alpha_num / alpha_den is compared exactly (alpha_num >= beta * alpha_den)."""
    if alpha_num >= cfg.beta * alpha_den:
        return d_init + cfg.l_d, k_init - cfg.l_k
    return d_init - cfg.l_d, k_init + cfg.l_k


def schedule(cfg: SchedCfg, left_record: Optional[Tuple[int, int]],
             prev: Optional[Tuple[int, int]], remaining: int) -> Tuple[int, int]:
    """(d_hat, k_hat) for the next tree.

    left_record: (d, k) recorded for the left neighbour cell, or None.
    prev: (accepted draft tokens a, depth d) of the previous tree (the acceptance statistic
          that drives Eq. 2), or None before the first tree.
    remaining: image tokens still to commit, the bonus token of this cycle included."""
    if left_record is None:
        d, k = cfg.d0, cfg.k0
    else:
        d, k = left_record
        if prev is not None and prev[1] > 0:
            d, k = bisect(d, k, prev[0], prev[1], cfg)
    d = clamp(d, cfg.d_lo, cfg.d_hi)
    k = clamp(k, cfg.k_lo, cfg.k_hi)
    d = min(d, remaining - 1)
    return d, k
