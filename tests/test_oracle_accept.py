"""Acceptance pins: greedy planted paths; the committed token's law under exact sampling
is p (Eq. 1 with point-mass proposals); relaxed mode reduces to exact mode at delta = 0."""
import numpy as np
import pytest

from oracle import accept as acc
from oracle.numerics import bf16_round


def _tree_with_chain(rng, chain_tokens, n_extra, V):
    """Tree whose chain root->c1->..->cm carries chain_tokens, plus distractor children with
    other tokens at random sibling ranks; BFS ordered."""
    parent, token, depth = [-1], [0], [0]
    chain_idx = [0]
    frontier = [0]
    for dpt, tok in enumerate(chain_tokens, start=1):
        sib = sorted(set(rng.choice([t for t in range(V) if t != tok], size=3, replace=False)))
        kids = sib[: rng.integers(0, 3)]
        pos = int(rng.integers(0, len(kids) + 1))
        kids = kids[:pos] + [tok] + kids[pos:]
        for t in kids:
            parent.append(chain_idx[-1])
            token.append(int(t))
            depth.append(dpt)
            if t == tok:
                mine = len(parent) - 1
        chain_idx.append(mine)
    return np.array(parent), np.array(token), chain_idx[1:]


def test_greedy_planted_path():
    rng = np.random.default_rng(0)
    V = 50
    for m in range(0, 6):
        target = rng.integers(0, V, size=m + 1)
        parent, token, chain = _tree_with_chain(rng, target[:m].tolist(), 3, V)
        n = len(parent)
        logits = rng.standard_normal((n, V))
        for j, u in enumerate([0] + chain):          # node u's argmax is the next chain token
            logits[u, target[j]] = 10.0
        path, bonus = acc.accept_greedy(logits, parent, token, np.tile([0, V], (n, 1)))
        assert path == chain and bonus == int(target[m])


def test_greedy_ties_and_allowed_range():
    logits = np.array([[1.0, 3.0, 3.0, 9.0]])
    assert acc.greedy_targets(logits, np.array([[0, 3]]))[0] == 1     # tie -> lowest id; id 3 not allowed


def _law_exact(w, sib_tokens):
    """Closed form of the committed token's law: sequential tries of the siblings, each
    accepted with (its weight)/(remaining weight), then a residual draw."""
    W = sum(w)
    rem = list(w)
    out = np.zeros(len(w))
    reach = 1.0
    for t in sib_tokens:
        Wr = sum(rem)
        out[t] += reach * rem[t] / Wr
        reach *= 1 - rem[t] / Wr
        rem[t] = 0
    Wr = sum(rem)
    out += reach * np.array(rem) / Wr
    return out


@pytest.mark.parametrize("sibs", [[], [2], [2, 0], [3, 1, 2]])
def test_exact_sampling_law_is_p(sibs):
    V = 5
    logits = np.array([0.3, -1.0, 1.2, 0.0, -0.4])
    w = acc.quantised_weights(logits, 0, V, 1.0, 0)
    p = np.array([int(x) for x in w], dtype=np.float64)
    p /= p.sum()
    assert np.allclose(_law_exact([int(x) for x in w], sibs), p, atol=1e-15)


def test_exact_sampling_histogram():
    """Committed first token over many seeds follows p (chi-square) for a 3-child root."""
    V = 6
    rng = np.random.default_rng(4)
    root_logits = rng.standard_normal(V)
    parent = np.array([-1, 0, 0, 0])
    token = np.array([0, 4, 1, 2])
    n = 4
    logits = np.vstack([root_logits, rng.standard_normal((n - 1, V))])
    allowed = np.tile([0, V], (n, 1))
    trials = 20_000
    counts = np.zeros(V)
    for s in range(trials):
        path, bonus = acc.accept_sampling(logits, parent, token, allowed, temperature=1.0, top_k=0,
                                          seed=1234, step=s, mode="exact")
        first = int(token[path[0]]) if path else bonus
        counts[first] += 1
    p = np.exp(root_logits - root_logits.max())
    p /= p.sum()
    chi2 = float(np.sum((counts - trials * p) ** 2 / (trials * p)))
    assert chi2 < 30.0                                      # 5 dof
    assert 0.5 * np.abs(counts / trials - p).sum() < 3 / np.sqrt(trials)


def test_top_k_truncation_and_temperature():
    logits = np.array([2.0, 1.0, 0.5, 3.0, -5.0])
    w = acc.quantised_weights(logits, 0, 5, 0.5, 2)
    assert [int(x) > 0 for x in w] == [True, False, False, True, False]
    assert int(w[3]) == 2 ** 32
    assert abs(int(w[0]) / 2 ** 32 - np.exp((2.0 - 3.0) / 0.5)) < 1e-6


def test_decision_boundary_is_exact(monkeypatch):
    """r < w_x accepts and r = w_x rejects (draws are stubbed)."""
    logits = np.array([[0.0, 0.0], [0.0, 0.0]])
    w = acc.quantised_weights(logits[0], 0, 2, 1.0, 0)
    wx = int(w[1])
    for r, accepted in ((wx - 1, True), (wx, False)):
        monkeypatch.setattr(acc, "draw_below", lambda u, W, r=r: r if W == 2 * wx else 0)
        path, _ = acc.accept_sampling(logits, [-1, 0], [0, 1], np.tile([0, 2], (2, 1)),
                                      temperature=1.0, top_k=0, seed=0, step=0)
        assert (path == [1]) == accepted


def test_relaxed_reduces_to_exact():
    rng = np.random.default_rng(5)
    V = 16
    knn = np.array([[x] + [int(y) for y in rng.permutation([t for t in range(V) if t != x])[:7]] for x in range(V)])
    parent = np.array([-1, 0, 0, 1, 1, 2])
    token = np.array([0, 3, 7, 1, 9, 3])
    logits = rng.standard_normal((6, V))
    allowed = np.tile([0, V], (6, 1))
    kw = dict(temperature=1.0, top_k=0, seed=9)
    for s in range(300):
        ex = acc.accept_sampling(logits, parent, token, allowed, step=s, mode="exact", **kw)
        assert acc.accept_sampling(logits, parent, token, allowed, step=s, mode="relaxed", delta=0.0,
                                   knn=knn, knn_k=8, **kw) == ex
        assert acc.accept_sampling(logits, parent, token, allowed, step=s, mode="relaxed", delta=0.3,
                                   knn=knn, knn_k=1, **kw) == ex


def test_relaxed_single_candidate_total_variation():
    """One drafted child x: the committed law is p with the credited neighbourhood mass moved
    onto x, so its total-variation distance to p is that mass, at most delta."""
    V = 8
    logits = np.array([0.5, 0.1, -0.3, 0.9, 0.0, -1.0, 0.4, 0.2])
    knn = np.array([[x] + [(x + j) % V for j in range(1, V)] for x in range(V)])
    x = 3
    delta = 0.25
    w = [int(v) for v in acc.quantised_weights(logits, 0, V, 1.0, 0)]
    W = sum(w)
    thr = (W * int(round(delta * 65536))) >> 16
    credit, extra = [], 0
    for y in knn[x][1:]:
        if extra + w[y] > thr:
            break
        extra += w[y]
        credit.append(int(y))
    law = np.zeros(V)
    law[x] = (w[x] + extra) / W
    rem = np.array(w, dtype=np.float64)
    rem[[x] + credit] = 0
    law += (1 - (w[x] + extra) / W) * rem / rem.sum()
    p = np.array(w) / W
    tv = 0.5 * np.abs(law - p).sum()
    assert tv <= delta + 1e-12 and abs(tv - extra / W) < 1e-12
    trials = 20_000
    counts = np.zeros(V)
    for s in range(trials):
        path, bonus = acc.accept_sampling(logits[None].repeat(2, 0), [-1, 0], [0, x], np.tile([0, V], (2, 1)),
                                          temperature=1.0, top_k=0, seed=3, step=s, mode="relaxed",
                                          delta=delta, knn=knn, knn_k=V)
        counts[x if path else bonus] += 1
    nz = law > 0
    chi2 = float(np.sum((counts[nz] - trials * law[nz]) ** 2 / (trials * law[nz])))
    assert chi2 < 30.0


def test_codebook_knn_by_angle():
    """Unit vectors at known angles on a circle: cosine order is angular distance."""
    theta = np.array([0.0, 0.1, 0.35, 1.0, 2.0, -0.05, 3.1])
    cb = np.stack([np.cos(theta), np.sin(theta)], axis=1) * np.array([[1.0], [2.0], [0.5], [3.0], [1.0], [1.5], [1.0]])
    knn = acc.codebook_knn(cb, 4)
    for x in range(len(theta)):
        d = np.abs((theta - theta[x] + np.pi) % (2 * np.pi) - np.pi)
        d[x] = np.inf
        assert knn[x, 0] == x and list(knn[x, 1:]) == list(np.argsort(d, kind="stable")[:3])


def test_quantised_exp_weight_is_rounded_exp():
    """The weights' exp (a fixed sequence of double operations) against the platform's
    float64 exp: w = rint(exp(d) 2^32) on a dense grid of float32 exponents in [-45, 0], apart
    from values within 1e-4 of a rounding tie; w(0) = 2^32, w = 0 below -40 and for -inf,
    and w never increases as d decreases."""
    import math
    d = (-np.linspace(0.0, 45.0, 1_500_001)).astype(np.float32)
    w = acc.quantised_exp_weight(d)
    ref = np.array([math.exp(float(x)) for x in d[::7]]) * 2.0 ** 32
    wr = w[::7]
    tie = np.abs(ref - np.floor(ref) - 0.5) < 1e-4
    assert np.all((wr == np.rint(ref)) | tie)
    assert np.all((wr == 0) == (d[::7] < -40) | (np.rint(ref) == 0))
    assert w[0] == 2.0 ** 32 and np.all(np.diff(w) <= 0)
    assert acc.quantised_exp_weight(np.float32([-np.inf, -40.5]))[:2].tolist() == [0.0, 0.0]


def test_quantised_exp_coefficients():
    """The Horner coefficients are ln(2)^j / j! and log2(e), to the last bit of a double
    (checked against the math module's ln 2, an independent route to the same values)."""
    import math
    for j, c in enumerate(acc.EXP2_COEF):
        exact = math.log(2.0) ** j / math.factorial(j)
        assert abs(c - exact) <= 4 * math.ulp(exact), j
    assert acc.LOG2E == 1.0 / math.log(2.0) or abs(acc.LOG2E - 1.0 / math.log(2.0)) <= math.ulp(acc.LOG2E)
    assert len(acc.EXP2_COEF) == 14
