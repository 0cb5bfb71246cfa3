"""Acceptance along a verified draft tree (Sec. 3.1, Eq. 1; Sec. 5.1 for T = 0).

Greedy (T = 0): walk from the root; at node u let t_u be the target's argmax over the
allowed ids (lowest id on ties); move to the child whose token is t_u while one exists.
The accepted path ends at u and t_u is the bonus token.

Exact sampling: Eq. 1 accepts a drafted token with probability min(1, p/q).  The
drafted children are deterministic top-k proposals, so q is read as a point mass on the
proposed token; the test becomes 'accept x with probability p(x)', and after a
rejection the residual distribution is p with x removed and renormalised.  Siblings are
tried in order (highest draft score first); if all are rejected the bonus is drawn from
the residual.  The committed token's law is exactly p.

Relaxed mode (config of the ADT-Tree+LANTERN rows, Tables I-II): a drafted token x is
also credited with the target mass of its nearest codebook neighbours, taken in
similarity order for as long as their summed mass stays within delta of the remaining
mass; x is accepted with probability (mass of x + credited mass), and on rejection the
whole credited neighbourhood is removed from the residual.  delta = 0 or one neighbour
reduces it to exact mode.

If a rejection empties the truncated support (possible when top_k is small) the bonus is
the top-1 id of p.

Numbers: p is quantised once per row to integer weights w = rint(exp(d) * 2^32), d = z - max z
with z = logit / T over the top-K allowed ids (z and d in float32, the precision the kernel
decides in), and exp(d) evaluated by a fixed sequence of IEEE double operations
(quantised_exp_weight), so that the integers do not depend on any library's exp; all later
arithmetic is exact integer.  A draw is
r = floor(U * W / 2^64) with U the 64 bits of Philox4x32-10 at key = seed and
counter = (step, node, trial, 0), and W the remaining total weight.

Literal Eq. 1 with stochastic children (accept_mss): the children of a node are i.i.d.
draws from q, so Eq. 1's ratio applies as printed.  Siblings are tried in draw order:
child x is accepted with probability min(1, p(x) / q(x)); after a rejection p becomes the
residual norm(max(0, p - q)) (the multi-step rule of SpecInfer, which the paper builds on)
and the next sibling is tried against it; if all are rejected the bonus is drawn from the
last residual, and at a leaf from p.  The committed token's law is exactly p.  Numbers: p
and q are the same integer weights as above (q from the draft row that drew the children),
with totals W_p, W_q; the test u < p(x)/q(x) with a 32-bit uniform u = U >> 32 is the
integer comparison u * q_w(x) * W_p < 2^32 * p_w(x) * W_q; the residual weights are
max(0, p_w(y) W_q - q_w(y) W_p) shifted right until the largest fits in 32 bits.

Test infrastructure only; see the package docstring.
"""
from __future__ import annotations

from typing import List, Optional, Sequence, Tuple

import numpy as np

from decimal import Decimal, getcontext

from .numerics import draw_below, uniform_u64

DELTA_FRAC_BITS = 16


def _exp2_coefficients(n: int = 14) -> Tuple[List[float], float]:
    """The doubles nearest ln(2)^j / j! (j < n), the Taylor coefficients of 2^f = e^(f ln 2),
    and the double nearest log2(e), from 60-digit decimal arithmetic (Decimal -> float rounds
    to nearest)."""
    getcontext().prec = 60
    ln2 = Decimal(2).ln()
    coef, fact = [], Decimal(1)
    for j in range(n):
        if j:
            fact *= j
        coef.append(float(ln2 ** j / fact))
    return coef, float(Decimal(1) / ln2)


EXP2_COEF, LOG2E = _exp2_coefficients()


def quantised_exp_weight(d: np.ndarray) -> np.ndarray:
    """w = rint(exp(d) * 2^32) for float32 exponents d <= 0, as float64 integers: y = d log2(e),
    k = floor(y), f = y - k in [0, 1), 2^f by Horner's rule over EXP2_COEF (degree 13, each
    step one rounded multiply then one rounded add), exp(d) = 2^f 2^k; d < -40 gives 0
    (exp(d) 2^32 < 2^-25).  Every step is an IEEE double operation, so an implementation that
    follows the same sequence without fused multiply-adds gets the same integers."""
    d64 = np.asarray(d, dtype=np.float32).astype(np.float64)
    live = d64 >= -40.0
    y = np.where(live, d64, 0.0) * LOG2E
    k = np.floor(y)
    f = y - k
    p = np.full_like(f, EXP2_COEF[-1])
    for c in EXP2_COEF[-2::-1]:
        p = p * f
        p = p + c
    w = np.rint(np.ldexp(p, (k + 32).astype(np.int64)))
    return np.where(live, w, 0.0)


def codebook_knn(codebook: np.ndarray, k: int) -> np.ndarray:
    """Neighbourhood of the relaxed mode: row x = x itself, then the k-1 other codes with the
    highest cosine similarity to code x (float64; ties to the lower id)."""
    c = np.asarray(codebook, dtype=np.float64)
    c = c / np.linalg.norm(c, axis=1, keepdims=True)
    sims = c @ c.T
    n = len(c)
    ids = np.arange(n)
    out = np.zeros((n, k), dtype=np.int32)
    for x in range(n):
        row = sims[x].copy()
        row[x] = -np.inf
        order = np.lexsort((ids, -row))[: k - 1]
        out[x, 0] = x
        out[x, 1:] = order
    return out


def greedy_targets(logits: np.ndarray, allowed: np.ndarray) -> np.ndarray:
    """t_u = argmax over [lo_u, hi_u) (np.argmax returns the lowest index among ties)."""
    out = np.zeros(len(logits), dtype=np.int64)
    for u in range(len(logits)):
        lo, hi = int(allowed[u][0]), int(allowed[u][1])
        out[u] = lo + int(np.argmax(logits[u][lo:hi]))
    return out


def children_of(parent: Sequence[int]) -> List[List[int]]:
    ch: List[List[int]] = [[] for _ in parent]
    for i in range(1, len(parent)):
        ch[int(parent[i])].append(i)
    return ch


def accept_greedy(logits: np.ndarray, parent, token, allowed) -> Tuple[List[int], int]:
    """Returns (accepted node indices v_1..v_a, bonus token)."""
    t = greedy_targets(logits, allowed)
    ch = children_of(parent)
    path: List[int] = []
    u = 0
    while True:
        nxt = [c for c in ch[u] if int(token[c]) == int(t[u])]
        if not nxt:
            return path, int(t[u])
        u = nxt[0]
        path.append(u)


def quantised_weights(logit_row: np.ndarray, lo: int, hi: int, temperature: float, top_k: int) -> np.ndarray:
    """Integer weights (Python ints in an object array) of the sampling distribution p at
    one row: softmax(logit / T) over the allowed ids, truncated to the top_k ids by
    (logit desc, id asc), as w = quantised_exp_weight(z - max z) with z in float32."""
    V = len(logit_row)
    z = np.asarray(logit_row[lo:hi], dtype=np.float32) / np.float32(temperature)
    ids = np.arange(lo, hi)
    keep = np.lexsort((ids, -z.astype(np.float64)))
    if top_k > 0:
        keep = keep[:top_k]
    zmax = z[keep].max()
    wq = quantised_exp_weight(z[keep] - zmax)               # float32 exponents
    w = np.zeros(V, dtype=object)
    w[:] = 0
    for i, val in zip(ids[keep], wq):
        w[int(i)] = int(val)
    return w


def top1_id(logit_row: np.ndarray, lo: int, hi: int, temperature: float) -> int:
    z = np.asarray(logit_row[lo:hi], dtype=np.float32) / np.float32(temperature)
    return lo + int(np.argmax(z))


def inverse_cdf(w: np.ndarray, r: int) -> int:
    """Smallest id i with sum_{j <= i} w_j > r (ids ascending)."""
    acc = 0
    for i in range(len(w)):
        acc += int(w[i])
        if acc > r:
            return i
    raise ValueError("draw beyond total weight")


def accept_sampling(logits: np.ndarray, parent, token, allowed, *, temperature: float, top_k: int,
                    seed: int, step: int, mode: str = "exact", delta: float = 0.0,
                    knn: Optional[np.ndarray] = None, knn_k: int = 1) -> Tuple[List[int], int]:
    """Exact (mode='exact') or relaxed (mode='relaxed') acceptance.  Returns (path, bonus)."""
    ch = children_of(parent)
    delta_q = int(round(delta * (1 << DELTA_FRAC_BITS)))
    path: List[int] = []
    u = 0
    while True:
        lo, hi = int(allowed[u][0]), int(allowed[u][1])
        w = quantised_weights(logits[u], lo, hi, temperature, top_k)
        W = int(sum(int(x) for x in w))
        accepted = None
        trial = 0
        for c in ch[u]:
            x = int(token[c])
            r = draw_below(uniform_u64(seed, step, u, trial), W)
            trial += 1
            credit = [x]
            mass = int(w[x])
            if mode == "relaxed" and x < len(knn):
                thr = (W * delta_q) >> DELTA_FRAC_BITS
                extra = 0
                for y in knn[x][1:knn_k]:
                    y = int(y)
                    if extra + int(w[y]) > thr:
                        break
                    extra += int(w[y])
                    credit.append(y)
                mass += extra
            if r < mass:
                accepted = c
                break
            for y in credit:
                W -= int(w[y])
                w[y] = 0
        if accepted is None:
            if W <= 0:
                # every id of the truncated support was removed: fall back to the top-1 id of p
                return path, top1_id(logits[u], lo, hi, temperature)
            r = draw_below(uniform_u64(seed, step, u, trial), W)
            return path, inverse_cdf(w, r)
        path.append(accepted)
        u = accepted


MSS_WEIGHT_BITS = 32


def accept_mss(logits: np.ndarray, q_rows: dict, parent, token, allowed, *, temperature: float, top_k: int,
               seed: int, step: int) -> Tuple[List[int], int]:
    """Multi-step acceptance of a tree with stochastic children (Eq. 1 with the residual
    norm(max(0, p - q))).  q_rows[u]: the draft logit row whose q drew node u's children.
    Returns (path, bonus)."""
    ch = children_of(parent)
    path: List[int] = []
    u = 0
    while True:
        lo, hi = int(allowed[u][0]), int(allowed[u][1])
        wp = [int(v) for v in quantised_weights(logits[u], lo, hi, temperature, top_k)]
        Wp = sum(wp)
        trial = 0
        accepted = None
        if ch[u]:
            wq = [int(v) for v in quantised_weights(q_rows[u], lo, hi, temperature, top_k)]
            Wq = sum(wq)
            for c in ch[u]:
                x = int(token[c])
                u32 = uniform_u64(seed, step, u, trial) >> 32
                trial += 1
                if u32 * wq[x] * Wp < (wp[x] * Wq) << 32:
                    accepted = c
                    break
                res = [max(0, wp[y] * Wq - wq[y] * Wp) for y in range(len(wp))]
                shift = max(0, max(res).bit_length() - MSS_WEIGHT_BITS)
                wp = [v >> shift for v in res]
                Wp = sum(wp)
                if Wp == 0:
                    # p == q on the support: a rejection has probability zero; kept for safety
                    return path, top1_id(logits[u], lo, hi, temperature)
        if accepted is None:
            r = draw_below(uniform_u64(seed, step, u, trial), Wp)
            return path, inverse_cdf(np.asarray(wp, dtype=object), r)
        path.append(accepted)
        u = accepted
