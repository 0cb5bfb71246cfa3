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
