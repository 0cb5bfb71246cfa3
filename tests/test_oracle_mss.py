"""Pins of the stochastic-children variant (Sec. 3.1 read literally: children sampled from
q, Eq. 1's min(1, p/q), residual norm(max(0, p - q))): closed forms of the acceptance
rates and of the committed token's law, checked by Monte Carlo over Philox counters, and
the structure of the sampled tree."""
import math

import numpy as np
import pytest

from oracle.accept import accept_mss, quantised_weights
from oracle.expand import build_tree, expand_sampled, sampled_children

V = 6
N_TRIALS = 12000


def _norm(w):
    w = np.asarray([float(x) for x in w])
    return w / w.sum()


def _logits(probs):
    return np.log(np.asarray(probs, dtype=np.float64)).astype(np.float32)


def _one_level(p_logits, q_logits, c, seed, step):
    """Root with c children drawn from q (leaves); returns (first committed token, accepted)."""
    ids, _ = sampled_children(q_logits, 0, V, c, 1.0, 0, seed, step, 0)
    parent = [-1] + [0] * c
    token = [7] + ids
    logits = np.stack([p_logits] + [p_logits] * c)
    path, bonus = accept_mss(logits, {0: q_logits}, parent, token, [(0, V)] * (c + 1), temperature=1.0, top_k=0,
                             seed=seed, step=step)
    return (token[path[0]] if path else bonus), bool(path)


def _binom_tol(p, n):
    return 5.0 * math.sqrt(max(p * (1 - p), 1e-4) / n) + 2e-3


@pytest.mark.parametrize("c", [1, 2, 3])
def test_committed_law_is_p_and_acceptance_matches_closed_form(c):
    """Disjoint-ish p and q: the committed token's frequencies equal p (SpecInfer's theorem),
    and the rate of accepting some child equals 1 - prod_j (1 - a_j) with a_1 = sum min(p, q),
    a_{j+1} = sum min(p_j, q), p_{j+1} = norm(max(0, p_j - q)).  The point-mass rule (accept
    x with probability p(x)) has the same law but a different rate (sum_x q(x) p(x) for one
    child), so the rate pins Eq. 1's ratio."""
    p_logits = _logits([0.45, 0.3, 0.1, 0.05, 0.05, 0.05])
    q_logits = _logits([0.05, 0.05, 0.1, 0.2, 0.3, 0.3])
    p = _norm(quantised_weights(p_logits, 0, V, 1.0, 0))
    q = _norm(quantised_weights(q_logits, 0, V, 1.0, 0))
    miss, pj = 1.0, p.copy()
    for _ in range(c):
        a = np.minimum(pj, q).sum()
        miss *= 1 - a
        r = np.maximum(pj - q, 0)
        pj = r / r.sum() if r.sum() > 0 else pj
    rate = 1 - miss
    point_mass_rate = float((q * p).sum())
    counts = np.zeros(V)
    acc = 0
    for t in range(N_TRIALS):
        tok, ok = _one_level(p_logits, q_logits, c, seed=11, step=t)
        counts[tok] += 1
        acc += ok
    freq = counts / N_TRIALS
    for x in range(V):
        assert abs(freq[x] - p[x]) <= _binom_tol(p[x], N_TRIALS), (x, freq, p)
    assert abs(acc / N_TRIALS - rate) <= _binom_tol(rate, N_TRIALS), (acc / N_TRIALS, rate)
    if c == 1:
        assert abs(rate - point_mass_rate) > 10 * _binom_tol(rate, N_TRIALS)


def test_equal_p_and_q_always_accept():
    """p == q: min(1, p/q) = 1, so the first child is accepted on every draw."""
    lg = _logits([0.3, 0.25, 0.2, 0.1, 0.1, 0.05])
    for t in range(500):
        _, ok = _one_level(lg, lg, 2, seed=3, step=t)
        assert ok


def test_point_mass_q_reduces_to_accepting_with_p():
    """q concentrated on one id x (every other logit far below): children are x, and the
    first is accepted with probability min(1, p(x) / 1) = p(x)."""
    p_logits = _logits([0.2, 0.35, 0.15, 0.1, 0.1, 0.1])
    q_logits = np.full(V, -200.0, dtype=np.float32)
    q_logits[1] = 0.0
    p = _norm(quantised_weights(p_logits, 0, V, 1.0, 0))
    acc = sum(_one_level(p_logits, q_logits, 1, seed=5, step=t)[1] for t in range(N_TRIALS))
    assert abs(acc / N_TRIALS - p[1]) <= _binom_tol(p[1], N_TRIALS)


def test_children_are_draws_from_q():
    """Drawn children follow q (temperature 0.7, top-4 truncation: truncated ids never drawn)."""
    rng = np.random.default_rng(8)
    lg = rng.normal(0, 1.5, V).astype(np.float32)
    q = _norm(quantised_weights(lg, 0, V, 0.7, 4))
    counts = np.zeros(V)
    n = 0
    for t in range(3000):
        ids, _ = sampled_children(lg, 0, V, 3, 0.7, 4, 21, t, 5)
        for i in ids:
            counts[i] += 1
            n += 1
    freq = counts / n
    for x in range(V):
        if q[x] == 0:
            assert counts[x] == 0
        else:
            assert abs(freq[x] - q[x]) <= _binom_tol(q[x], n)


def test_sampled_tree_structure_and_budget():
    """Every drawn child is kept; layer sizes follow the budget rule (k_hat nodes expanded
    while whole expansions fit); BFS order is creation order, so siblings are contiguous in
    draw order and a node's tree index is its pool index + 1; deterministic per counter."""
    rng = np.random.default_rng(4)
    Vb = 40
    table = rng.normal(0, 2.0, (64, Vb)).astype(np.float32)
    calls = []

    def level_fn(frontier, pool):
        calls.append(list(frontier))
        return np.stack([table[(pool[u].token * 7 + u) % 64] for u in frontier])

    kw = dict(temperature=1.0, top_k=0, seed=9, step=4)
    pool, sel = expand_sampled(table[0], level_fn, 3, 2, 3, 20, lambda d: (0, Vb), **kw)
    # layer 1: 3; depth 2: min(2, 3, (20-3)//3) = 2 expanded -> 6; depth 3: min(2, 6, (20-9)//3) = 2 -> 6
    assert len(pool) == 15 and sel == list(range(15))
    assert [len(c) for c in calls] == [2, 2]
    depths = [nd.depth for nd in pool]
    assert depths == [1] * 3 + [2] * 6 + [3] * 6
    tree = build_tree(5, pool, sel, by_creation=True)
    for i in range(1, tree.n):
        assert tree.pool_index[i] == i - 1
        par = pool[i - 1].parent
        assert tree.parent[i] == (0 if par < 0 else par + 1)
    # frontier = best two of the previous layer by (score desc, creation asc)
    lay1 = sorted(range(3), key=lambda c: (-pool[c].score, c))[:2]
    assert calls[0] == lay1
    # same counters, same tree; another step, another draw somewhere
    calls.clear()
    pool2, _ = expand_sampled(table[0], level_fn, 3, 2, 3, 20, lambda d: (0, Vb), **kw)
    assert [(a.token, a.parent) for a in pool2] == [(a.token, a.parent) for a in pool]
    kw["step"] = 5
    pool3, _ = expand_sampled(table[0], level_fn, 3, 2, 3, 20, lambda d: (0, Vb), **kw)
    assert [a.token for a in pool3] != [a.token for a in pool]
    # a budget that admits no second layer
    pool4, _ = expand_sampled(table[0], level_fn, 3, 2, 3, 5, lambda d: (0, Vb), **kw)
    assert len(pool4) == 3


def test_oracle_decode_with_stochastic_children():
    """The decoder in stochastic-children mode on the tiny model: every expanded node has
    exactly c children, trees stay within the budget, siblings are contiguous (draw order),
    committed tokens lie in their cells' allowed ranges, and the run is deterministic."""
    import dataclasses
    import synth
    from oracle.decode import Decoder
    from oracle.model import OracleModel
    cfg = synth.get_config("tiny")
    cfg = dataclasses.replace(cfg, accept=synth.AcceptCfg(mode="mss", temperature=1.0, top_k=0, children=3))
    w = synth.model_weights(cfg)
    om = OracleModel(cfg, w)
    pre = synth.prefix_ids(cfg)
    runs = []
    for _ in range(2):
        dec = Decoder(cfg, om, pre)
        dec.prefill()
        out = []
        for _ in range(6):
            info = dec.step()
            tr = info.tree
            kids = {}
            for i in range(1, tr.n):
                kids.setdefault(int(tr.parent[i]), []).append(i)
            for u, ks in kids.items():
                assert len(ks) == 3 and ks == list(range(ks[0], ks[0] + 3))
            assert tr.n - 1 <= cfg.sched.n_budget
            for j, tok in enumerate(info.committed):
                lo, hi = cfg.allowed(info.L_before + 1 + j - len(pre))
                assert lo <= tok < hi
            out.append((tr.token.tolist(), info.committed))
        runs.append(out)
    assert runs[0] == runs[1]
