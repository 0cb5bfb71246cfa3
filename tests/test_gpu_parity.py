"""Layer-local and cross-fed parity of the HIP path with the oracle at the benchmarked shapes:
LlamaGen-XL (36 layers, d 1280, V 16384, greedy), Lumina-mGPT-7B (32 layers, d 4096, V 65536,
row-end tokens, Poisson-driven schedule, greedy) and Anole-7B (exact and relaxed sampling over
8192 image codes), all at full depth, at the stated tolerances.

Floating point, layer by layer.  The session records (adt_session_set_capture) the residual
stream entering every decoder layer of every forward it runs -- prefill chunks, draft catch-up
rows, draft frontier levels, verify -- plus each forward's tokens, positions, ancestor masks and
the draft head's FC input rows.  The oracle then evaluates each half of each layer (the
attention block with its output projection, the SwiGLU block; Sec. 3.1 and the draft head of
Sec. 4.2 / Fig. 5) from the GPU's own input to that half, against the GPU's own K/V cache for the
keys it reads, and every result must lie within |gpu - oracle| <= 2e-2 + 1e-2 |oracle| element
by element: the half's contribution to the residual, the residual after it, the K and V rows the
layer appends, the draft FC output, the final features and the logits (the LM head from the
GPU's final features).  An error inside any one layer therefore shows up at that layer, however
deep; rounding differences carried in from earlier layers do not accumulate in the comparison.

Integers, cross-fed.  Each cycle the GPU decodes its own trajectory and the oracle re-decides
every integer decision from the GPU's own floating-point outputs: the schedule (Eq. 2) from the
GPU's acceptance history (it must also equal the library's host schedule); the expansion
(Eq. 3-5: top-k, frontier selection, rerank, BFS tree) from the GPU's draft logits; the
acceptance (greedy argmax walk, or the exact / relaxed sampling walk with the shared Philox
draws) from the GPU's verify logits; the KV compaction of the GPU's pre-commit cache rows.
Trees, paths, bonus tokens, committed tokens and compacted rows must be bit-exact.  The only
exception: where the GPU's fp32 path scores (sums of logit - log-sum-exp) order two candidates
whose fp64 scores are closer than the observed score error, the two orders are both correct;
such a frontier or rerank boundary is accepted only with that margin, and counted.  Because the
oracle follows the GPU's trajectory, the comparison never stops at a divergence.
"""
import dataclasses
import gc
import time

import numpy as np
import pytest
import torch

import synth
from oracle import accept as acc
from oracle.decode import compact_cache
from oracle.expand import build_tree, expand
from oracle.model import KVCache, OracleModel
from oracle.numerics import masked_logits, rmsnorm
from oracle.schedule import initial, schedule

pytestmark = pytest.mark.gpu

TOL = (2e-2, 1e-2)
T0 = time.time()


def log(*a):
    print(f"[{time.time() - T0:7.1f}s]", *a, flush=True)


@pytest.fixture(scope="module")
def rt():
    from paper_2512_21857_amd import runtime
    assert torch.cuda.is_available()
    return runtime


def f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().to(torch.float32).cpu().numpy().astype(np.float64)


class Report:
    def __init__(self, name):
        self.name = name
        self.worst = {}
        self.fail = []
        self.count = {}

    def check(self, what, got, ref, where=""):
        got = np.asarray(got, dtype=np.float64)
        ref = np.asarray(ref, dtype=np.float64)
        assert got.shape == ref.shape, (what, got.shape, ref.shape)
        if ref.size == 0:
            return
        ratio = np.abs(got - ref) / (TOL[0] + TOL[1] * np.abs(ref))
        w = float(ratio.max())
        if not np.isfinite(w):
            w = float("inf")
        self.worst[what] = max(self.worst.get(what, 0.0), round(w, 4))
        if w > 1.0:
            i = np.unravel_index(int(np.argmax(ratio)), ratio.shape)
            self.fail.append(f"{what} {where}: worst |diff|/tol {w:.3f} at {i} (gpu {got[i]:.6g}, oracle {ref[i]:.6g})")

    def exact(self, what, ok, detail=""):
        self.count[what] = self.count.get(what, 0) + 1
        if not ok:
            self.fail.append(f"{what}: {detail}")

    def bump(self, what):
        self.count[what] = self.count.get(what, 0) + 1

    def summary(self):
        return {"config": self.name, "worst_ratio": self.worst, "counts": self.count, "failures": self.fail[:20]}


def _bits(mask_row):
    out = []
    for w in range(2):
        word = int(mask_row[w])
        j = 0
        while word:
            if word & 1:
                out.append(64 * w + j)
            word >>= 1
            j += 1
    return out


def _cache_layer(t: torch.Tensor) -> np.ndarray:
    """[H][S][Dh] bf16 device cache slice -> float64 host copy."""
    return f64(t)


# ------------------------------------------------------------------------------ layer-local
def _caches(sess, draft, nb, layers):
    """[branch][layer] (K, V) device views of the session's caches."""
    if draft:
        return [[(sess.dk_cache[b] if nb > 1 else sess.dk_cache, sess.dv_cache[b] if nb > 1 else sess.dv_cache)]
                for b in range(nb)]
    return [[((sess.k_cache[b] if nb > 1 else sess.k_cache)[l], (sess.v_cache[b] if nb > 1 else sess.v_cache)[l])
             for l in range(layers)] for b in range(nb)]


def check_forward(rep, om, sess, rec, what, nb=1):
    """The oracle evaluates every half-layer of one recorded forward from the GPU's inputs,
    branch by branch (with guidance, node r's branch-b row is row nb r + b).  Returns the
    oracle's final norm of the GPU's last residual, [branch][rows][d]."""
    m = om.m
    n, d = rec["nodes"], m.d_model
    assert rec["rows"] == n * nb
    pos = [int(p) for p in rec["pos"]]
    Lp, s0 = rec["kv_prefix"], rec["slot0"]
    slots = [s0 + r for r in range(n)]
    keys = [list(range(Lp)) + [Lp + j for j in _bits(rec["mask"][r])] for r in range(n)]
    for r in range(n):
        assert slots[r] in keys[r], f"{what}: row {r} does not see its own slot"
    Rall = f64(rec["resid"])
    names = ["draft"] if rec["draft"] else [f"layer{l}" for l in range(m.n_layers)]
    caches = _caches(sess, rec["draft"], nb, m.n_layers)
    out = []
    for b in range(nb):
        R = Rall[:, b::nb]
        tag_b = what + (f" branch {b}" if nb > 1 else "")
        # the tokens recorded are branch 0's; every branch shares them outside the prompt
        same_tok = b == 0 or not what.startswith("prefill")
        if rec["draft"]:
            xin = f64(rec["xin"])[b::nb]
            if same_tok:
                rep.exact(f"{what}: FC input embedding half", np.array_equal(xin[:, :d], om.embed_rows(rec["tok"])),
                          "embedding rows differ")
            rep.check("draft FC output", R[0], xin @ om.w("draft.fc").T, tag_b)
        elif same_tok:
            rep.exact(f"{what}: embedding", np.array_equal(R[0], om.embed_rows(rec["tok"])), "embedding rows differ")
        for li, pre in enumerate(names):
            kc = f64(caches[b][li][0])
            vc = f64(caches[b][li][1])
            H, S, Dh = kc.shape
            cache = KVCache(1, H, S, Dh)
            cache.k[0] = kc
            cache.v[0] = vc
            h_in, h_mid, h_out = R[2 * li], R[2 * li + 1], R[2 * li + 2]
            o_mid, _, _ = om.attn_block(pre, h_in, pos, slots, keys, cache, 0)
            tag = f"{tag_b} {pre}"
            rep.check("attention block contribution", h_mid - h_in, o_mid - h_in, tag)
            rep.check("residual after attention", h_mid, o_mid, tag)
            rep.check("K rows appended", kc[:, slots, :], cache.k[0][:, slots, :], tag)
            rep.check("V rows appended", vc[:, slots, :], cache.v[0][:, slots, :], tag)
            o_out, _, _ = om.mlp_block(pre, h_mid)
            rep.check("MLP block contribution", h_out - h_mid, o_out - h_mid, tag)
            rep.check("layer output", h_out, o_out, tag)
        out.append(om.rnd(rmsnorm(R[-1])))
    return out


def check_head(rep, om, feat_gpu, logits_gpu, f_ref, what, scale=None, branch_logits=None, cols=None):
    """Final features (per branch) against the oracle's norm of the GPU's final residual;
    logits against the oracle's LM head applied to the GPU's own features, over the vocabulary
    columns cols = (lo, hi) the session computes (the union of the cells' allowed ranges).
    With guidance the per-branch logits (when given) are checked, and the guided logits
    l_u + s (l_c - l_u) against the branch logits' combination within the propagated bound
    (|1 - s| + s) tol."""
    nb = len(f_ref)
    base = []
    for b in range(nb):
        if feat_gpu is not None:
            rep.check("final features", feat_gpu[b], f_ref[b], what)
            base.append(feat_gpu[b])
        else:
            base.append(f_ref[b])
    if logits_gpu is None:
        return
    lo, hi = cols if cols is not None else (0, logits_gpu.shape[-1])
    lb = [(x @ om.w("lm_head").T)[..., lo:hi] for x in base]
    logits_gpu = logits_gpu[..., lo:hi]
    if branch_logits is not None:
        branch_logits = [x[..., lo:hi] for x in branch_logits]
    if nb == 1:
        rep.check("logits", logits_gpu, lb[0], what)
        return
    if branch_logits is not None:
        for b in range(nb):
            rep.check("branch logits", branch_logits[b], lb[b], what)
    ref = lb[1] + scale * (lb[0] - lb[1])
    k = abs(1.0 - scale) + scale
    bound = k * (TOL[0] + TOL[1] * np.maximum(np.abs(lb[0]), np.abs(lb[1])))
    ratio = float(np.max(np.abs(logits_gpu - ref) / bound))
    rep.worst["guided logits / propagated bound"] = max(rep.worst.get("guided logits / propagated bound", 0.0),
                                                       round(ratio, 4))
    if ratio > 1.0:
        rep.fail.append(f"guided logits {what}: {ratio:.3f} of the propagated bound")


def _ws_rows(sess, ptr, rows, cols, dtype):
    return sess._ws(ptr, rows * cols, dtype).view(rows, cols)


# ------------------------------------------------------------------------------ cross-fed integers
def crossfed_expand(rep, cfg, t, level_recs, L, root_token, d_hat, k_hat, n_budget, P):
    """The oracle's expansion on the GPU's draft logits must rebuild the GPU's tree."""
    dl = f64(t["draft_logits"])
    k_hi = cfg.sched.k_hi
    levels = []

    def level_fn(frontier, pool):
        lvl = len(levels) + 2
        levels.append([int(pool[u].token) for u in frontier])
        base = 1 + (lvl - 2) * k_hi
        return dl[base: base + len(frontier)]

    allowed_at = lambda depth: cfg.allowed(L + depth - P)
    pool, sel = expand(dl[0], level_fn, d_hat, k_hat, n_budget, allowed_at)
    ot = build_tree(root_token, pool, sel)
    gp = t["parent"].cpu().numpy()
    gt = t["token"].cpu().numpy()
    gs = t["score"].cpu().numpy().astype(np.float64)

    def paths(parent, token):
        out = []
        for i in range(len(parent)):
            p, u = [], i
            while u > 0:
                p.append(int(token[u]))
                u = int(parent[u])
            out.append(tuple(reversed(p)))
        return out

    og, oo = paths(gp, gt), paths(ot.parent, ot.token)
    score_of = {pth: float(s) for pth, s in zip(oo, ot.score)}
    errs = [abs(gs[i] - score_of[pth]) for i, pth in enumerate(og) if pth in score_of]
    err = max(errs) if errs else 0.0
    rep.worst["score |gpu - oracle|"] = max(rep.worst.get("score |gpu - oracle|", 0.0), err)
    rep.exact("score error below 1e-4", err <= 1e-4, f"{err}")
    eps = max(2.0 * err, 1e-6)
    # frontier tokens of every level against the GPU's level forwards
    g_levels = [[int(x) for x in r["tok"]] for r in level_recs]

    def level_gap(depth):
        sc = sorted((c.score for c in pool if c.depth == depth), reverse=True)
        return sc[k_hat - 1] - sc[k_hat] if len(sc) > k_hat else np.inf

    for i, (o, g) in enumerate(zip(levels, g_levels)):
        if o != g:
            gap = level_gap(i + 1)
            rep.exact("frontier differs only at an fp32 score near-tie", gap < eps,
                      f"level {i + 2}: oracle {o} gpu {g}, boundary gap {gap:.3g} >= {eps:.3g}")
            rep.bump("frontier near-tie")
            return ot
    if len(levels) != len(g_levels):
        rep.exact("expansion levels", False, f"oracle {len(levels)} gpu {len(g_levels)}")
        return ot
    from oracle.tree import packed_mask
    rep.exact("tree masks and depths", np.array_equal(t["mask"].cpu().numpy().view(np.uint64), packed_mask(gp, 2)) and
              t["depth"].cpu().tolist() == [len(pth) for pth in og], "")
    if og == oo and gp.tolist() == ot.parent.tolist():
        rep.bump("trees bit-exact")
        return ot
    if set(og) != set(oo):
        ranked = sorted((c.score for c in pool), reverse=True)
        gap = ranked[n_budget - 1] - ranked[n_budget] if len(ranked) > n_budget else np.inf
        rep.exact("rerank differs only at an fp32 score near-tie", gap < eps,
                  f"selected sets differ, boundary gap {gap:.3g} >= {eps:.3g}")
        rep.bump("rerank near-tie")
        return ot
    # same nodes, another BFS order: every swapped pair must be an fp32 near-tie at one depth
    pos_o = {pth: i for i, pth in enumerate(oo)}
    perm = [pos_o[pth] for pth in og]
    for a in range(len(perm)):
        for b in range(a + 1, len(perm)):
            if perm[a] > perm[b]:
                sa, sb = score_of[og[a]], score_of[og[b]]
                ok = len(og[a]) == len(og[b]) and abs(sa - sb) < eps
                rep.exact("BFS order differs only at fp32 score near-ties", ok,
                          f"nodes {og[a]} / {og[b]} scores {sa:.9g} / {sb:.9g}")
    rep.bump("BFS order near-tie")
    return ot


def crossfed_accept(cfg, knn, logits, parent, token, allowed, step):
    masked = np.stack([masked_logits(logits[i], *allowed[i]) for i in range(len(parent))])
    a = cfg.accept
    if a.mode == "greedy":
        return acc.accept_greedy(masked, parent, token, allowed)
    return acc.accept_sampling(masked, parent, token, allowed, temperature=a.temperature, top_k=a.top_k,
                               seed=cfg.seed, step=step, mode=a.mode, delta=a.delta, knn=knn, knn_k=a.knn_k)


# ------------------------------------------------------------------------------ the run
def run_parity(rt, cfg, dm, om, n_cycles, poisson=None, knn=None, fixed_tree=False):
    """Layer-local float checks and cross-fed integer checks over n_cycles cycles of the GPU's
    own trajectory (fixed_tree: every cycle (d_hi, k_hi) instead of the schedule)."""
    m = cfg.model
    d, V, P = m.d_model, m.vocab, cfg.prefix_len
    guided = cfg.guidance is not None
    nb = 2 if guided else 1
    gs = cfg.guidance
    rep = Report(cfg.name + ("" if cfg.accept.mode == "greedy" else f"/{cfg.accept.mode}") +
                 (f"/guided {gs}" if guided else "") + ("/fixed" if fixed_tree else ""))
    knn_t = torch.from_numpy(knn).cuda() if knn is not None else None
    sess = rt.DeviceSession(dm, cfg, poisson=poisson, knn=knn_t, fixed_tree=fixed_tree)
    tdt = torch.bfloat16 if m.dtype == "bf16" else torch.float32
    sess.set_capture(resid_elems=(2 * m.n_layers + 1) * 128 * d + 8 * 128 * 3 * d, xin_bytes=4 * 128 * 2 * d * 4,
                     meta_elems=1 << 16)
    pre = synth.prefix_ids(cfg)
    null = synth.null_prefix_ids(cfg) if guided else None
    first = sess.prefill(pre, null)
    recs = sess.captured()
    v = sess.view()
    f_ref = None
    for r in recs:
        if r["draft"]:
            check_forward(rep, om, sess, r, f"prefill draft rows {r['slot0']}..", nb)
        else:
            f_ref = check_forward(rep, om, sess, r, f"prefill target rows {r['slot0']}..", nb)
    # the last chunk's features and the last prompt row's logits
    last = recs[-2] if recs[-1]["draft"] else recs[-1]
    assert not last["draft"]
    cn = last["nodes"]
    feat = f64(_ws_rows(sess, v.feat, cn * nb, d, tdt)).reshape(cn, nb, d)
    lg = f64(_ws_rows(sess, v.logits, 1, V, torch.float32))
    bl = f64(_ws_rows(sess, v.branch_logits, nb, V, torch.float32)) if guided else None
    check_head(rep, om, [feat[:, b] for b in range(nb)], None, f_ref, "prefill")
    check_head(rep, om, [feat[cn - 1: cn, b] for b in range(nb)], lg[0:1], [f[cn - 1: cn] for f in f_ref],
               "prefill last row", gs, None if bl is None else [bl[b: b + 1] for b in range(nb)],
               cols=(v.logits_lo, v.logits_hi))
    gfeat = [{} for _ in range(nb)]   # GPU target features (bf16 values as float64) per committed position
    for r in range(cn):
        for b in range(nb):
            gfeat[b][last["slot0"] + r] = feat[r, b]
    lo, hi = cfg.allowed(0)
    op, ob = crossfed_accept(cfg, knn, lg, [-1], [int(pre[-1])], [(lo, hi)], 0)
    rep.exact("first token (cross-fed)", op == [] and ob == first, f"oracle {ob} gpu {first}")
    log(rep.name, "prefill checked", {k: v for k, v in rep.worst.items()})
    records, prev, prev_cell = {}, None, None
    sched = rt.sched_struct(cfg.sched, cfg.grid_w)
    for cyc in range(1, n_cycles + 1):
        v = sess.view()
        L, Ld, step = v.L, v.Ld, v.step
        tokens = [v.tokens_host[i] for i in range(v.n_tokens)]
        cell = L + 1 - P
        remaining = cfg.n_image - cell
        if remaining <= 0:
            break
        if fixed_tree:
            d_hat, k_hat = min(cfg.sched.d_hi, remaining - 1), cfg.sched.k_hi
        else:
            # schedule from the GPU's history: the oracle's and the library's host rule agree
            pv = prev
            if pv is not None and cfg.sched.alpha_source == "poisson":
                pv = (min(int(poisson[prev_cell]), pv[1]), pv[1])
            init = initial(cfg.sched, cell, records, cfg.grid_w)
            d_hat, k_hat = schedule(cfg.sched, init, pv, remaining)
            c_init = rt.schedule_init(sched, cell, records, cfg.n_image)
            c_dk = rt.schedule_next(sched, c_init, pv, remaining)
            rep.exact("schedule (oracle = library host rule)", (d_hat, k_hat) == c_dk, f"{(d_hat, k_hat)} vs {c_dk}")
        if d_hat >= 1:
            sess.restart_capture()
            sess.expand(d_hat, k_hat, cfg.sched.n_budget)
            drecs = sess.captured()
            assert all(r["draft"] for r in drecs)
            t = sess.tensors()
            # catch-up rows: the FC input's feature half is the GPU's target feature of p - 1
            cu = drecs[0]
            xin = f64(cu["xin"])
            for r, p in enumerate(cu["pos"]):
                p = int(p)
                for b in range(nb):
                    if p - 1 in gfeat[b]:
                        rep.exact("catch-up FC input feature = committed target feature",
                                  np.array_equal(xin[nb * r + b, d:], gfeat[b][p - 1]), f"position {p} branch {b}")
            fr = check_forward(rep, om, sess, cu, f"cycle {cyc} draft catch-up", nb)
            dl = f64(t["draft_logits"])
            dbl = f64(t["draft_branch_logits"]) if guided else None
            check_head(rep, om, None, dl[0:1], [f[-1:] for f in fr], f"cycle {cyc} draft root", gs,
                       None if dbl is None else [dbl[b: b + 1] for b in range(nb)], cols=t["logits_range"])
            for li, r in enumerate(drecs[1:]):
                fr = check_forward(rep, om, sess, r, f"cycle {cyc} draft level {li + 2}", nb)
                base = 1 + li * cfg.sched.k_hi
                check_head(rep, om, None, dl[base: base + r["nodes"]], fr, f"cycle {cyc} draft level {li + 2}", gs,
                           cols=t["logits_range"])
            crossfed_expand(rep, cfg, t, drecs[1:], L, tokens[L], d_hat, k_hat, cfg.sched.n_budget, P)
        else:
            sess.set_tree([-1], [tokens[L]])
        sess.restart_capture()
        sess.verify()
        vrec = sess.captured()
        assert len(vrec) == 1 and not vrec[0]["draft"]
        t = sess.tensors()
        n = t["n"]
        f_ref = check_forward(rep, om, sess, vrec[0], f"cycle {cyc} verify", nb)
        feat = f64(t["feat"]).reshape(n, nb, d)
        logits32 = t["logits"].cpu().numpy()
        vbl = f64(t["branch_logits"]) if guided else None
        check_head(rep, om, [feat[:, b] for b in range(nb)], logits32.astype(np.float64), f_ref, f"cycle {cyc} verify",
                   gs, None if vbl is None else [vbl[:, b] for b in range(nb)], cols=t["logits_range"])
        parent = t["parent"].cpu().numpy()
        token = t["token"].cpu().numpy()
        depth = t["depth"].cpu().numpy()
        allowed = t["allowed"].cpu().numpy()
        want_allowed = np.array([cfg.allowed(L + int(dp) + 1 - P) for dp in depth])
        rep.exact("allowed ranges of the tree rows", np.array_equal(allowed, want_allowed), "")
        # pre-commit K/V rows of the tree, every layer (and branch)
        pk = f64(sess.k_cache[..., L: L + n, :])
        pvv = f64(sess.v_cache[..., L: L + n, :])
        opath, obonus = crossfed_accept(cfg, knn, logits32, parent, token, allowed, step)
        g = sess.accept_commit(d_hat, k_hat)
        t2 = sess.tensors()
        a = g["n_accepted"]
        gpath = t2["path"][1: a + 1].cpu().tolist() if a else []
        rep.exact("accepted path (cross-fed)", gpath == list(opath), f"cycle {cyc}: oracle {opath} gpu {gpath}")
        rep.exact("bonus token (cross-fed)", g["tokens"][-1] == obonus, f"cycle {cyc}: oracle {obonus} gpu {g['tokens'][-1]}")
        rep.exact("committed tokens", g["tokens"] == [int(token[u]) for u in gpath] + [g["tokens"][-1]], "")
        # compaction: slot L + m <- slot L + v_m, bit for bit
        ck, cv = pk.copy(), pvv.copy()
        compact_cache(ck, cv, 0, gpath)
        post_k = f64(sess.k_cache[..., L: L + 1 + a, :])
        post_v = f64(sess.v_cache[..., L: L + 1 + a, :])
        rep.exact("compacted K/V rows", np.array_equal(post_k, ck[..., : a + 1, :]) and
                  np.array_equal(post_v, cv[..., : a + 1, :]), f"cycle {cyc}")
        rep.exact("draft cache length after the cycle", sess.view().Ld == (L + 1 if d_hat >= 1 else Ld), "")
        for b in range(nb):
            gfeat[b][L] = feat[0, b]
            for mm, u in enumerate(gpath, start=1):
                gfeat[b][L + mm] = feat[u, b]
        for c in range(cell, cell + a + 1):
            records[c] = (d_hat, k_hat)
        prev, prev_cell = (a, d_hat), cell
        rep.bump("cycles")
        log(rep.name, f"cycle {cyc}: d={d_hat} k={k_hat} n={n} a={a}", {k: v for k, v in rep.worst.items()})
    sess.set_capture(0)
    del sess
    gc.collect()
    torch.cuda.empty_cache()
    s = rep.summary()
    log(s)
    return s


def _models(rt, cfg):
    log(cfg.name, "generating weights")
    w = synth.model_weights(cfg, threads=16)
    dm = rt.DeviceModel(cfg, w)
    log(cfg.name, "model on the GPU")
    om = OracleModel(cfg, w, cache_f64=True)
    return w, dm, om


def test_llamagen_xl_full_shape_parity(rt):
    """The LlamaGen-XL shape (36 layers, d 1280, 20 x 64 heads, FFN 3584, V 16384, 120-token
    prompt in two prefill chunks, greedy): 10 cycles at full depth under the ADT schedule."""
    cfg = synth.get_config("llamagen_xl")
    w, dm, om = _models(rt, cfg)
    s = run_parity(rt, cfg, dm, om, 10)
    assert not s["failures"], s
    assert s["counts"]["cycles"] >= 8


def test_lumina_7b_full_depth_parity(rt):
    cfg = synth.get_config("lumina_7b")
    w, dm, om = _models(rt, cfg)
    s = run_parity(rt, cfg, dm, om, 8, poisson=synth.poisson_table(cfg))
    assert not s["failures"], s
    assert s["counts"]["cycles"] >= 8


def test_anole_7b_full_depth_parity_exact_and_relaxed(rt):
    """Exact (tree rejection sampling) and relaxed (k = 100 codebook neighbours, delta = 0.1)
    acceptance on the same model; both sides use the oracle's neighbour table (the GPU's own
    table is compared separately)."""
    from oracle.accept import codebook_knn
    cfg = synth.get_config("anole_7b", mode="exact")
    w, dm, om = _models(rt, cfg)
    s = run_parity(rt, cfg, dm, om, 8)
    assert not s["failures"], s
    rcfg = synth.get_config("anole_7b", mode="relaxed")
    knn = codebook_knn(synth.codebook(rcfg), 100)
    s2 = run_parity(rt, rcfg, dm, om, 8, knn=knn)
    assert not s2["failures"], s2
    assert s["counts"]["cycles"] >= 8 and s2["counts"]["cycles"] >= 8


def _small_bf16():
    cfg = synth.shrink(synth.get_config("llamagen_xl"), n_layers=2, d_model=256, n_heads=4, ffn=512, vocab=512)
    return dataclasses.replace(cfg, prefix_len=16, img_hi=512, prefix_hi=512, grid_h=8, grid_w=8)


@pytest.mark.parametrize("variant", ["adt", "fixed", "guided", "subrange", "subrange_high"])
def test_bf16_small_parity(rt, variant):
    """The 2-layer bf16 model (d 256, 4 x 64 heads, V 512, 8 x 8 grid) under the ADT schedule,
    with fixed 6-deep 10-wide trees, with classifier-free guidance (scale 3.0), and with image
    ids [64, 320) inside the vocabulary (the LM head then computes those 256 rows only, from
    weight row 64 on); and with V 8192 and image ids [2500, 6000), so that the root's and each
    level's top-k cover only the 2048-id chunks 1-2 of the row, starting at a 16-unaligned id:
    every cycle of the image layer-local within the bf16 tolerance and cross-fed bit-exact."""
    cfg = _small_bf16()
    if variant == "guided":
        cfg = dataclasses.replace(cfg, guidance=3.0)
    if variant == "subrange":
        cfg = dataclasses.replace(cfg, img_lo=64, img_hi=320, prefix_lo=320, prefix_hi=512)
    if variant == "subrange_high":
        cfg = synth.shrink(synth.get_config("llamagen_xl"), n_layers=2, d_model=256, n_heads=4, ffn=512, vocab=8192)
        cfg = dataclasses.replace(cfg, prefix_len=16, img_lo=2500, img_hi=6000, prefix_lo=6000, prefix_hi=8192,
                                  grid_h=8, grid_w=8)
    w = synth.model_weights(cfg)
    dm = rt.DeviceModel(cfg, w)
    om = OracleModel(cfg, w)
    s = run_parity(rt, cfg, dm, om, 64, fixed_tree=variant == "fixed")
    assert not s["failures"], s
    assert s["counts"]["cycles"] >= 8
