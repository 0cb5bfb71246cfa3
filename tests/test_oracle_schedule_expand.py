"""Schedule (Sec. 4.1-4.2, Eq. 2) and expansion (Sec. 3.1, Sec. 4.2, Eq. 3-5) pins."""
import json
import math
import os

import numpy as np
import pytest

from synth import SchedCfg
from oracle.expand import build_tree, expand, pool_size
from oracle.schedule import schedule

GOLD = os.path.join(os.path.dirname(__file__), "golden")


@pytest.mark.parametrize("case", json.load(open(os.path.join(GOLD, "schedule_trajectories.json")))["cases"],
                         ids=lambda c: c["name"][:20])
def test_schedule_trajectories(case):
    cfg = SchedCfg(**case["sched"])
    rec, prev = None, None
    got = []
    for a in case["accepted"][: len(case["trees"])]:
        d, k = schedule(cfg, rec, prev, remaining=10_000)
        got.append([d, k])
        rec, prev = (d, k), (a, d)
    assert got == case["trees"]


def test_schedule_end_of_image_and_first_tree():
    cfg = SchedCfg(1, 6, 4, 10, 1, 10, 1.0, 60, 5, 10)
    assert schedule(cfg, None, None, remaining=3) == (2, 10)
    assert schedule(cfg, (6, 4), (6, 6), remaining=1) == (0, 4)        # last token: plain AR step


def _depth_q(gold):
    return {int(k): np.log(np.array(v)) for k, v in gold["q_by_depth"].items()}


def _run_golden(gold, n_budget):
    q = _depth_q(gold)
    level_fn = lambda frontier, pool: np.stack([q[pool[u].depth + 1] for u in frontier])
    return expand(q[1], level_fn, gold["d_hat"], gold["k_hat"], n_budget, lambda d: (0, 4))


def test_expand_golden_pool_and_trees():
    gold = json.load(open(os.path.join(GOLD, "expand_small.json")))
    for case in gold["cases"]:
        pool, sel = _run_golden(gold, case["n_budget"])
        assert [p.token for p in pool] == gold["pool_tokens"]
        assert np.allclose([math.exp(p.score) for p in pool], gold["pool_prob"], rtol=1e-12)
        assert len(pool) == pool_size(gold["d_hat"], gold["k_hat"])
        t = build_tree(7, pool, sel)
        assert t.parent.tolist() == case["parent"]
        assert t.token[1:].tolist() == case["token"] and t.token[0] == 7
        assert t.depth.tolist() == case["depth"]
        assert np.allclose(np.exp(t.score), case["prob"], rtol=1e-12)


def _hashed_level(V, seed):
    """Draft logits that depend only on (node token, depth): a fixed hash, no model."""
    def row(token, depth):
        return np.random.default_rng([seed, token, depth]).standard_normal(V) * 2.0
    return row


@pytest.mark.parametrize("d_hat,k_hat,N", [(1, 4, 16), (3, 4, 16), (4, 3, 60), (6, 10, 60), (2, 13, 60)])
def test_expand_invariants(d_hat, k_hat, N):
    V = 37
    row = _hashed_level(V, 11)
    root = row(5, 0)
    level_fn = lambda frontier, pool: np.stack([row(pool[u].token, pool[u].depth) for u in frontier])
    pool, sel = expand(root, level_fn, d_hat, k_hat, N, lambda d: (0, V))
    assert len(pool) == pool_size(d_hat, k_hat)                      # Eq. 5
    assert len(sel) == min(N, len(pool))
    t = build_tree(5, pool, sel)                                     # raises unless ancestor-closed
    for i in range(1, t.n):
        assert 0 <= t.parent[i] < i and t.depth[i] == t.depth[t.parent[i]] + 1
        assert t.score[i] <= t.score[t.parent[i]]                    # log q <= 0 along a path
    scores = sorted([p.score for p in pool], reverse=True)
    assert sorted(t.score[1:].tolist(), reverse=True) == scores[: len(sel)]   # top-N of the pool
    # frontier rule: only the k best nodes of each layer have children
    for depth in range(1, d_hat):
        layer = sorted([p for p in pool if p.depth == depth], key=lambda p: (-p.score, p.creation))
        parents = {p.parent for p in pool if p.depth == depth + 1}
        assert parents == {p.creation for p in layer[:k_hat]}
    # siblings carry distinct tokens, ordered by draft rank
    for u in range(t.n):
        kids = [i for i in range(1, t.n) if t.parent[i] == u]
        assert len({int(t.token[i]) for i in kids}) == len(kids)


def test_expand_restricted_vocab():
    """A depth whose allowed range holds one id gives every expanded node one child."""
    row = _hashed_level(20, 3)
    level_fn = lambda frontier, pool: np.stack([row(pool[u].token, pool[u].depth) for u in frontier])
    allowed = lambda d: (19, 20) if d == 2 else (0, 19)
    pool, sel = expand(row(1, 0), level_fn, 3, 4, 60, allowed)
    assert [p.token for p in pool if p.depth == 2] == [19] * 4
    assert sum(p.depth == 3 for p in pool) == 4 * 4


# ---------------------------------------------------------------- initialisation rules
# Sec. 4.1 (Horizontal / Vertical Repeat, Random), Sec. 5.3 (TokenFlock, Eqs. 6-8; the fixed
# bases of Table V) and the width rule at the end of Sec. 4.2.  Expected values below are
# worked by hand from those definitions.
def _cfg(**kw):
    import dataclasses
    return dataclasses.replace(SchedCfg(1, 6, 4, 10, 1, 10, 1.0, 60, 5, 10), **kw)


def test_horizontal_and_vertical_repeat():
    from oracle.schedule import initial
    W = 4
    rec = {g: (g % 6 + 1, g + 3) for g in range(1, 7)}          # cell 0 (prefill) has no record
    h, v = _cfg(), _cfg(init="vertical")
    assert initial(h, 7, rec, W) == rec[6]                     # left neighbour
    assert initial(v, 7, rec, W) == rec[3]                     # cell above (row 0, column 3)
    assert initial(v, 6, rec, W) == rec[2]
    assert initial(v, 2, rec, W) == rec[1]                     # first row: the left neighbour
    assert initial(v, 4, rec, W) == rec[3]                     # above = cell 0 has no record
    assert initial(h, 1, {}, W) is None and initial(v, 1, {}, W) is None


def test_tokenflock_hand_computed():
    from oracle.schedule import initial
    W, cell = 8, 28                                             # (y, x) = (3, 4)
    inside = {26: (2, 4), 27: (3, 5),                          # dy = 0, |dx| <= 2: weight 3
              19: (4, 6), 20: (5, 7), 21: (6, 8),              # dy = 1, |dx| <= 1: weight 2
              12: (1, 9)}                                       # dy = 2, dx = 0:    weight 1
    outside = {18: (30, 30), 22: (30, 30), 10: (30, 30), 4: (30, 30), 29: (30, 30)}
    cfg = _cfg(init="tokenflock", flock_delta=2)
    # d: (3*2 + 3*3 + 2*4 + 2*5 + 2*6 + 1*1) / 13 = 46/13 = 3.54 -> 4; k: 78/13 = 6
    assert initial(cfg, cell, {**inside, **outside}, W) == (4, 6)
    # delta = 1: left (weight 2) and above (weight 1) only: d = (2*3 + 5)/3 = 3.67 -> 4,
    # k = (2*5 + 7)/3 = 5.67 -> 6
    assert initial(_cfg(init="tokenflock", flock_delta=1), cell, {**inside, **outside}, W) == (4, 6)
    assert initial(_cfg(init="tokenflock", flock_delta=1), cell, {27: (3, 5), 20: (6, 8)}, W) == (4, 6)
    assert initial(_cfg(init="tokenflock", flock_delta=1), cell, {27: (3, 5), 20: (9, 11)}, W) == (5, 7)
    # equal weights, mean exactly half way: rounded up
    assert initial(_cfg(init="tokenflock", flock_delta=2), 2, {0: (1, 4), 1: (2, 7)}, W) == (2, 6)
    # constant records reproduce the constant; no recorded cell in range: no source
    assert initial(cfg, cell, {g: (3, 7) for g in range(cell)}, W) == (3, 7)
    assert initial(cfg, cell, {0: (3, 7)}, W) is None


def test_random_init_uniform_and_deterministic():
    from oracle.schedule import initial
    cfg = _cfg(init="random", seed=1234)
    n = 7000
    draws = [initial(cfg, c, {}, 16) for c in range(n)]
    assert draws == [initial(cfg, c, {c - 1: (9, 9)}, 16) for c in range(n)]   # records are ignored
    for col, lo, span in ((0, 1, 6), (1, 4, 7)):
        counts = np.bincount([t[col] - lo for t in draws], minlength=span)
        assert len(counts) == span
        exp = n / span
        assert float(np.sum((counts - exp) ** 2 / exp)) < 30.0          # <= 6 dof, p ~ 1e-4
    pairs = np.zeros((6, 7))
    for d, k in draws:
        pairs[d - 1, k - 4] += 1
    exp = n / 42
    assert float(np.sum((pairs - exp) ** 2 / exp)) < 90.0              # 41 dof: d and k independent
    other = [initial(_cfg(init="random", seed=1235), c, {}, 16) for c in range(64)]
    assert other != draws[:64]


def test_fixed_bases_table5():
    from oracle.schedule import initial
    rec = {3: (6, 10)}
    assert initial(_cfg(fix_d=1), 4, rec, 16) == (1, 10)
    assert initial(_cfg(fix_k=25), 4, rec, 16) == (6, 25)
    assert initial(_cfg(fix_d=1, fix_k=25), 4, rec, 16) == (1, 25)
    assert initial(_cfg(fix_d=1), 1, {}, 16) == (1, 10)                # first tree: (1, k0)
    cfg = _cfg(fix_d=1, fix_k=25)
    # negative: Eq. 2 gives (0, 35), clamped to (1, 10); positive: (2, 15) -> (2, 10)
    assert schedule(cfg, initial(cfg, 4, rec, 16), (0, 3), 100) == (1, 10)
    assert schedule(cfg, initial(cfg, 4, rec, 16), (3, 3), 100) == (2, 10)


def test_width_clamp_only_for_deep_trees():
    deep, always = _cfg(k_clamp="deep"), _cfg()
    # negative from (1, 10): adapted depth 0 -> width 20 kept up to 16 under the deep rule
    assert schedule(deep, (1, 10), (0, 1), 100) == (1, 16)
    assert schedule(always, (1, 10), (0, 1), 100) == (1, 10)
    assert schedule(deep, (2, 10), (1, 2), 100) == (1, 16)            # 2 - 1 = 1: not above 1
    assert schedule(deep, (1, 3), (0, 1), 100) == (1, 13)
    assert schedule(deep, (2, 10), (2, 2), 100) == (3, 4)             # depth 3: bounds apply
    assert schedule(deep, (1, 4), (1, 1), 100) == (2, 4)
    assert schedule(deep, (1, 3), None, 100) == (1, 3)                # no adaptation: d~ = 1
