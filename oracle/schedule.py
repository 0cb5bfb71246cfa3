"""Tree depth and width per cycle (Sec. 4): an initial (d~, k~) (Sec. 4.1: Horizontal Repeat,
Vertical Repeat, Random; Sec. 5.3: TokenFlock, Eqs. 6-8, and the fixed bases of Table V)
followed by bisectional dynamic adaptation (Sec. 4.2, Eq. 2) and the bounds of Sec. 4.2.

Readings where the paper is silent:
  * the record of an image cell is the (depth, width) of the tree whose cycle committed it;
    cell (i, j) is i * grid_w + j in raster order;
  * Horizontal Repeat takes the record of cell (i, j-1); at j = 0 the raster predecessor is
    used, and the first tree (no record yet) takes (d0, k0) without adaptation;
  * Vertical Repeat takes the record of cell (i-1, j); in the first row (and wherever that
    cell has no record) it falls back to Horizontal Repeat;
  * Random draws d~ and k~ uniformly from the inclusive depth and width bounds, for every
    tree, with one Philox4x32-10 block per cell: key = seed, counter = (cell, 0, 0, 1);
    the two 64-bit words (x1 x0) and (x3 x2) give floor(U * span / 2^64);
  * TokenFlock: x is the column and y the row; the set holds the recorded cells c < cell
    within Euclidean distance delta; norm() divides each weight (delta - dy + 1) / delta by
    the sum over the set; d~ and k~ are the weighted means rounded half up to integers; an
    empty set means no source ((d0, k0) without adaptation);
  * a fixed base replaces d~ (or k~) by its constant for every tree, the first included;
    Eq. 2 and the bounds then apply as usual;
  * the width bound is applied always, or (the "deep" rule) only when the adapted depth
    d~ +- l_d exceeds 1; a one-layer tree then keeps its width in [1, 16], 16 being the
    widest top-k one expansion layer supports (the paper gives no bound, and without one
    the width would grow by l_k on every negative one-layer cycle);
  * the acceptance rate is alpha = a / d, a counting accepted draft tokens only, so with
    beta = 1 a tree is 'positive' iff every drafted layer was accepted;
  * the bounds are inclusive ranges applied after Eq. 2, to depth and width alike;
  * near the end of the image the depth is cut to the tokens that remain minus one
    (the bonus token), and a depth of 0 means a plain AR step.

Test infrastructure only; see the package docstring.
"""
from __future__ import annotations

import math
from fractions import Fraction
from typing import Dict, Optional, Tuple

from synth import SchedCfg
from .numerics import MASK32, draw_below, philox4x32_10


def clamp(x: int, lo: int, hi: int) -> int:
    return max(lo, min(hi, x))


def bisect(d_init: int, k_init: int, alpha_num: int, alpha_den: int, cfg: SchedCfg) -> Tuple[int, int]:
    """Eq. 2: deeper and narrower when alpha >= beta, shallower and wider otherwise.
    alpha = alpha_num / alpha_den is compared exactly (alpha_num >= beta * alpha_den)."""
    if alpha_num >= cfg.beta * alpha_den:
        return d_init + cfg.l_d, k_init - cfg.l_k
    return d_init - cfg.l_d, k_init + cfg.l_k


MAX_WIDTH = 16


def _random_init(cfg: SchedCfg, cell: int) -> Tuple[int, int]:
    x0, x1, x2, x3 = philox4x32_10((cell, 0, 0, 1), (cfg.seed & MASK32, (cfg.seed >> 32) & MASK32))
    d = cfg.d_lo + draw_below((x1 << 32) | x0, cfg.d_hi - cfg.d_lo + 1)
    k = cfg.k_lo + draw_below((x3 << 32) | x2, cfg.k_hi - cfg.k_lo + 1)
    return d, k


def _token_flock(cfg: SchedCfg, cell: int, records: Dict[int, Tuple[int, int]], grid_w: int):
    """Eqs. 6-8 over the recorded past cells."""
    yi, xi = divmod(cell, grid_w)
    delta = cfg.flock_delta
    omega = []
    for c, rec in records.items():
        yj, xj = divmod(c, grid_w)
        if c < cell and math.sqrt((xi - xj) ** 2 + (yi - yj) ** 2) <= delta:
            omega.append((Fraction(delta - (yi - yj) + 1, delta), rec))
    if not omega:
        return None
    total = sum(w for w, _ in omega)
    d = sum(w / total * rd for w, (rd, _) in omega)
    k = sum(w / total * rk for w, (_, rk) in omega)
    half_up = lambda q: math.floor(q + Fraction(1, 2))
    return half_up(d), half_up(k)


def initial(cfg: SchedCfg, cell: int, records: Dict[int, Tuple[int, int]], grid_w: int):
    """(d~, k~) for the cycle whose first drafted token is image cell `cell`, or None (no
    source: the first tree).  records: cell -> (d, k) of every committed cell."""
    if cfg.init == "horizontal":
        init = records.get(cell - 1)
    elif cfg.init == "vertical":
        init = records.get(cell - grid_w) if cell >= grid_w else None
        if init is None:
            init = records.get(cell - 1)
    elif cfg.init == "random":
        init = _random_init(cfg, cell)
    elif cfg.init == "tokenflock":
        init = _token_flock(cfg, cell, records, grid_w)
    else:
        raise ValueError(cfg.init)
    if cfg.fix_d or cfg.fix_k:
        d, k = init if init is not None else (cfg.d0, cfg.k0)
        init = (cfg.fix_d or d, cfg.fix_k or k)
    return init


def schedule(cfg: SchedCfg, left_record: Optional[Tuple[int, int]],
             prev: Optional[Tuple[int, int]], remaining: int) -> Tuple[int, int]:
    """(d_hat, k_hat) for the next tree.

    left_record: the initial (d~, k~) (the left neighbour's record under Horizontal Repeat,
          otherwise what initial() returns), or None.
    prev: (accepted draft tokens a, depth d) of the previous tree (the acceptance statistic
          that drives Eq. 2), or None before the first tree.
    remaining: image tokens still to commit, the bonus token of this cycle included."""
    if left_record is None:
        d, k = cfg.d0, cfg.k0
    else:
        d, k = left_record
        if prev is not None and prev[1] > 0:
            d, k = bisect(d, k, prev[0], prev[1], cfg)
    if cfg.k_clamp == "deep":
        assert cfg.d_lo == 1
        k = clamp(k, 1, MAX_WIDTH) if d <= 1 else clamp(k, cfg.k_lo, cfg.k_hi)
    else:
        k = clamp(k, cfg.k_lo, cfg.k_hi)
    d = clamp(d, cfg.d_lo, cfg.d_hi)
    d = min(d, remaining - 1)
    return d, k
