"""GPU parity at the 7B shapes (Lumina-mGPT-shaped: row-end tokens, Poisson-driven schedule;
Anole-shaped: exact and relaxed sampling over 8192 image codes) against the fp64 oracle.

Per layer, at the real width and vocabulary (one-layer models of the same shapes): prefill,
draft and verify logits within the bf16 tolerance (2e-2, 1e-2) element by element, over
several ADT cycles with the schedule, trees and committed tokens compared exactly until the
first flagged near-tie.

At full depth the GPU (fp32 accumulation, bf16 storage) and the oracle (fp64, the same bf16
storage points) round the occasional value to neighbouring bf16 numbers, and RMSNorm carries
those one-ulp differences into the next layer; the logit difference therefore grows with
depth (measured: median |diff| 0.0029 at one layer, 0.0215 at 32 layers of the Lumina shape,
about layers^0.58).  An fp32 evaluation of the oracle on the CPU (fp32 BLAS, the same bf16
storage points) lands at similar distances from the fp64 oracle: one layer, prefill worst
|diff|/tol 0.63-0.85, draft logits 1.5-1.7 over three summation orders, against 0.83 and
2.2 for the GPU, whose one-layer target feature differs from fp64 by an RMS 1.4x that of
fp32 BLAS.  Logits are therefore checked against 1.5 * depth^0.6 times the tolerance,
depth being the number of decoder layers behind the value (the draft head's logits: the
target's layers plus its FC and its own layer, since it reads the target's bf16 feature),
and one-layer runs must have 99 % of the elements inside the plain tolerance.  Integer
decisions are compared until the first flagged near-tie."""
import gc

import numpy as np
import pytest
import torch

import synth
from oracle.accept import codebook_knn
from oracle.decode import Decoder
from oracle.expand import build_tree
from oracle.model import OracleModel

pytestmark = pytest.mark.gpu

TOL = (2e-2, 1e-2)


@pytest.fixture(scope="module")
def rt():
    from paper_2512_21857_amd import runtime
    assert torch.cuda.is_available()
    return runtime


def _check(got, ref, depth, what, report, one_layer):
    """Elementwise bound 1.5 * depth^0.6 times the tolerance (depth = decoder layers behind the
    value; 1.5 = headroom for the GPU's fp32 arithmetic, whose one-layer feature deviates from
    fp64 1.4x as much, in RMS, as fp32 BLAS does); for one-layer models also at least 99 % of
    the elements inside the plain tolerance (98 % for the draft head, three rounding stages
    deep: a single normalised input element that fp32 and fp64 round to neighbouring bf16
    values moves that row's K and V by one ulp in ~17 % of their elements, and every later
    row attends to it).  Returns the largest absolute difference."""
    tol = TOL[0] + TOL[1] * np.abs(ref)
    diff = np.abs(got - ref)
    ratio = diff / tol
    inside = float((ratio <= 1.0).mean())
    rec = report.setdefault(what, {"worst_ratio": 0.0, "min_inside_plain": 1.0})
    rec["worst_ratio"] = max(rec["worst_ratio"], round(float(ratio.max()), 3))
    rec["min_inside_plain"] = min(rec["min_inside_plain"], round(inside, 5))
    assert ratio.max() <= 1.5 * float(depth) ** 0.6, f"{what}: worst |diff|/tol {ratio.max():.3f} at depth {depth}"
    if one_layer:
        need = 0.99 if depth <= 1 else 0.98
        assert inside >= need, f"{what}: only {inside:.4f} inside the plain tolerance"
    return float(diff.max())


def _near_tie(sorted_vals, upto, err):
    """True when two of the first upto+1 values of a descending list are closer than 2*err,
    i.e. when an order or membership decision among them may go either way at error err."""
    v = np.asarray(sorted_vals[: upto + 1])
    return bool(len(v) > 1 and np.min(v[:-1] - v[1:]) < 2.0 * err)


def _shared_logit_accept(rt, sess, logits, parent, token, allowed, step, path, bonus):
    """The session's acceptance kernel on the oracle's logits (cast to fp32, the precision both
    sides decide in) must reproduce the oracle's accepted path and bonus exactly."""
    dev = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a, dtype=dt)).cuda()
    n = len(parent)
    gpath, gn, gb = rt.verify_accept(dev(logits, np.float32), dev(parent, np.int32), dev(token, np.int32),
                                     dev(allowed, np.int32), dev([n], np.int32), sess.accept, step)
    a = int(gn.item())
    assert gpath[1:a + 1].cpu().tolist() == list(path) and int(gb.item()) == bonus, "shared-logit acceptance differs"


def _side_by_side(rt, cfg, n_steps, knn_g=None, knn_o=None, poisson=None):
    """Each cycle: the oracle schedules and expands; the GPU expands with the same (d, k) (draft
    logits compared; the first tree level compared exactly unless the oracle's own top-k margin
    is inside the observed error); both then verify, accept and commit the oracle's tree (verify
    logits compared; the acceptance kernel re-decides the oracle's logits bit for bit; greedy
    commits compared exactly unless the oracle's argmax margin at the deciding node is inside
    the observed error).  After an accepted divergence the oracle runs the remaining cycles
    alone, each acceptance still re-decided by the GPU kernel on the oracle's logits."""
    n_l = cfg.model.n_layers
    one = n_l == 1
    greedy = cfg.accept.mode == "greedy"
    print(f"[{cfg.name}] generating weights", flush=True)
    w = synth.model_weights(cfg, threads=16)
    dm = rt.DeviceModel(cfg, w)
    om = OracleModel(cfg, w, cache_f64=True)
    pre = synth.prefix_ids(cfg)
    sess = rt.DeviceSession(dm, cfg, poisson=poisson, knn=knn_g)
    dec = Decoder(cfg, om, pre, poisson=poisson, knn=knn_o)
    print(f"[{cfg.name}] prefill", flush=True)
    g_first = sess.prefill(pre)
    o_first = dec.prefill()
    # the prefill's last-row logits sit in row 0 of the logits buffer
    gp = sess.tensors()["logits"][0].cpu().numpy()
    err = np.abs(gp - dec.prefill_logits)
    report = {"first_equal": g_first == o_first, "steps": 0, "flag": None, "layers": n_l,
              "prefill_max_err": float(err.max()), "prefill_median_err": float(np.median(err)),
              "tree_level1_ties": 0, "deeper_tree_differs": 0}
    e_pre = _check(gp, dec.prefill_logits, n_l, "prefill", report, one)
    print(f"[{cfg.name}] {report}", flush=True)
    _shared_logit_accept(rt, sess, dec.prefill_logits[None], [-1], [int(pre[-1])], [dec.allowed_pos(dec.P)], 0, [],
                         o_first)
    if g_first != o_first:
        lo, hi = dec.allowed_pos(dec.P)
        z = np.sort(dec.prefill_logits[lo:hi])[::-1]
        if greedy:
            assert _near_tie(z, 1, e_pre), "first token differs without a near-tie"
        else:
            assert lo <= g_first < hi
        report["flag"] = "first token differs (near-tie)" if greedy else "first token differs (sampling near-boundary)"
    matched = 0
    while report["flag"] is None and matched < n_steps and not dec.done():
        d, k = dec.schedule_next()
        print(f"[{cfg.name}] cycle {matched + 1}: d={d} k={k}", flush=True)
        if d >= 1:
            tree, droot = dec.expand_tree(d, k)
            n = sess.expand(d, k, cfg.sched.n_budget)
            t = sess.tensors()
            e_d = _check(t["draft_logits"][0].cpu().numpy(), droot, n_l + 2, "draft_logits", report, one)
            gp_, gt_ = t["parent"].cpu().numpy(), t["token"].cpu().numpy()
            g1 = [int(gt_[i]) for i in range(n) if gp_[i] == 0]
            o1 = [int(tree.token[i]) for i in range(tree.n) if tree.parent[i] == 0]
            # property: the GPU's first level is the top-k of its own root draft row
            lo, hi = dec.allowed_pos(dec.L + 1)
            gz = t["draft_logits"][0].cpu().numpy()[lo:hi]
            order = np.lexsort((np.arange(hi - lo), -gz.astype(np.float64)))
            assert g1 == [lo + int(i) for i in order[:len(g1)]], "first level is not the top-k of its draft row"
            if g1 != o1:
                lo, hi = dec.allowed_pos(dec.L + 1)
                z = np.sort(droot[lo:hi])[::-1]
                assert _near_tie(z, k, e_d), f"first tree level differs without a near-tie: {g1} vs {o1}"
                report["tree_level1_ties"] += 1
            elif n != tree.n or gp_.tolist() != tree.parent.tolist() or gt_.tolist() != tree.token.tolist():
                report["deeper_tree_differs"] += 1
            info_tree = tree
        else:
            info_tree = build_tree(dec.tokens[-1], [], [])
            droot = None
        sess.set_tree(info_tree.parent.tolist(), info_tree.token.tolist())
        sess.verify()
        gl = sess.tensors()["logits"].cpu().numpy()
        info = dec.verify_commit(info_tree, d, k, expanded=d >= 1, draft_root=droot)
        _check(gl, info.logits, n_l, "verify_logits", report, one)
        _shared_logit_accept(rt, sess, info.logits, info_tree.parent, info_tree.token, info.allowed, info.step,
                             info.path, info.bonus)
        g = sess.accept_commit(d, k)
        if g["tokens"] != info.committed:
            j = next(i for i in range(min(len(g["tokens"]), len(info.committed)))
                     if g["tokens"][i] != info.committed[i])
            v = 0 if j == 0 else int(info.path[j - 1])
            lo, hi = info.allowed[v]
            if greedy:
                row_err = float(np.abs(gl[v] - info.logits[v]).max())
                z = np.sort(info.logits[v][lo:hi])[::-1]
                assert _near_tie(z, 1, row_err), f"commit differs at node {v} without a near-tie"
            else:
                # a valid walk of the same tree: committed drafts follow a root path, the last
                # token lies in its row's allowed range
                cur = 0
                for tok in g["tokens"][:-1]:
                    kids = [i for i in range(info_tree.n) if info_tree.parent[i] == cur and info_tree.token[i] == tok]
                    assert kids, "GPU committed a token that is not a child on its path"
                    cur = kids[0]
                blo, bhi = info.allowed[cur]
                assert blo <= g["tokens"][-1] < bhi
            report["flag"] = f"committed tokens differ at cycle {matched + 1} (near-tie)" if greedy else \
                f"committed tokens differ at cycle {matched + 1} (sampling near-boundary)"
            break
        matched += 1
    report["steps"] = matched
    # past a divergence the oracle decodes alone; its every acceptance is re-decided by the
    # GPU kernel on the same fp32 logits and trees
    report["oracle_only_accept_checks"] = 0
    while matched + report["oracle_only_accept_checks"] < n_steps and not dec.done():
        info = dec.step()
        _shared_logit_accept(rt, sess, info.logits, info.tree.parent, info.tree.token, info.allowed, info.step,
                             info.path, info.bonus)
        report["oracle_only_accept_checks"] += 1
    print(f"[{cfg.name}] {report}", flush=True)
    del sess, dm
    gc.collect()
    torch.cuda.empty_cache()
    return report


@pytest.mark.parametrize("layers", [1, None], ids=["one_layer", "full_depth"])
def test_lumina_7b_cycles(rt, layers):
    cfg = synth.get_config("lumina_7b")
    if layers:
        cfg = synth.shrink(cfg, n_layers=layers)
    rep = _side_by_side(rt, cfg, 4 if layers else 3, poisson=synth.poisson_table(cfg))
    print("lumina", rep)
    assert rep["flag"] is None or "near-tie" in rep["flag"] or "near-boundary" in rep["flag"]


@pytest.mark.parametrize("layers", [1, None], ids=["one_layer", "full_depth"])
def test_anole_7b_exact_cycles(rt, layers):
    cfg = synth.get_config("anole_7b", mode="exact")
    if layers:
        cfg = synth.shrink(cfg, n_layers=layers)
    rep = _side_by_side(rt, cfg, 4 if layers else 3)
    print("anole exact", rep)
    assert rep["flag"] is None or "near-tie" in rep["flag"] or "near-boundary" in rep["flag"]


def test_codebook_knn_matches_oracle(rt):
    """Cosine top-100 of the 8192 x 256 codebook: each row starts with the code itself and holds
    distinct ids; rows equal the oracle's, except where the oracle's own similarity gap at the
    first differing rank is below what an fp32 dot product resolves."""
    cfg = synth.get_config("anole_7b", mode="relaxed")
    cb = synth.codebook(cfg)
    g = rt.codebook_knn(torch.from_numpy(cb).cuda(), 100).cpu().numpy()
    o = codebook_knn(cb, 100)
    c = cb.astype(np.float64)
    c /= np.linalg.norm(c, axis=1, keepdims=True)
    assert (g[:, 0] == np.arange(len(cb))).all()
    assert all(len(set(r)) == len(r) for r in g.tolist())
    bad, worst = 0, 0.0
    for x in np.nonzero((g != o).any(axis=1))[0]:
        j = int(np.argmax(g[x] != o[x]))
        gap = abs(float(c[x] @ c[o[x, j]]) - float(c[x] @ c[g[x, j]]))
        assert gap < 1e-6, f"row {x} rank {j}: gap {gap}"
        bad += 1
        worst = max(worst, gap)
    print(f"knn rows differing at near-ties: {bad}, largest similarity gap {worst:.3g}")
    # adjacent similarities of the top 100 among 8191 random directions are ~4e-4 apart, an
    # fp32 dot of 256 terms is good to ~1e-7: expect well under 1 % of rows to swap a pair
    assert bad <= len(cb) // 100


def test_anole_7b_relaxed_cycles(rt):
    """Relaxed mode (one layer at the real width) with the oracle's neighbour table given to both
    sides (the GPU table is checked separately above)."""
    cfg = synth.shrink(synth.get_config("anole_7b", mode="relaxed"), n_layers=1)
    ko = codebook_knn(synth.codebook(cfg), 100)
    rep = _side_by_side(rt, cfg, 4, knn_g=torch.from_numpy(ko).cuda(), knn_o=ko)
    print("anole relaxed", rep)
    assert rep["flag"] is None or "near-tie" in rep["flag"] or "near-boundary" in rep["flag"]
