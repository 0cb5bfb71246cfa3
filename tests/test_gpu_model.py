"""GPU parity of whole cycles (adt_step / adt_tree_expand / adt_verify_forward /
adt_session_accept_commit) against the oracle decoder on the same seeded model.

Integer outputs (schedule, tree arrays, accepted paths, committed tokens) must match bit
for bit.  Where a floating-point comparison decides an integer, the GPU (fp32 or bf16
arithmetic) and the oracle (fp64) may legitimately pick different winners when the
oracle's own margin is below the float tolerance; such a decision is a flagged near-tie,
reported, and the trajectory comparison stops there (both continue from different
states).  Logits and features: (1e-5, 1e-5) in fp32, (2e-2, 1e-2) in bf16."""
import dataclasses

import numpy as np
import pytest
import torch

import synth
from oracle.decode import Decoder, ar_decode
from oracle.expand import Tree
from oracle.model import OracleModel
from oracle.tree import depths

pytestmark = pytest.mark.gpu

TOL = {"f32": (1e-5, 1e-5), "bf16": (2e-2, 1e-2)}


def _tol_ok(got, ref, tol):
    return np.abs(got - ref) <= tol[0] + tol[1] * np.abs(ref)


@pytest.fixture(scope="module")
def rt():
    from paper_2512_21857_amd import runtime
    assert torch.cuda.is_available()
    return runtime


def _setup(rt, cfg, **sess_kw):
    w = synth.model_weights(cfg)
    om = OracleModel(cfg, w)
    dm = rt.DeviceModel(cfg, w)
    pre = synth.prefix_ids(cfg)
    return w, om, dm, pre


def _greedy_margin(row, lo, hi):
    seg = np.sort(np.asarray(row[lo:hi], dtype=np.float64))
    return seg[-1] - seg[-2] if len(seg) > 1 else np.inf


def _guided_ok(got, ref, branch_refs, s, tol):
    """Guided logits u + s (c - u): each branch within tol moves them by at most
    (|1 - s| + s) (atol + rtol max(|c|, |u|))."""
    k = abs(1.0 - s) + s
    scale = np.maximum(np.abs(branch_refs[0]), np.abs(branch_refs[1]))
    return np.abs(got - ref) <= k * (tol[0] + tol[1] * scale)


def _compare_run(rt, cfg, n_steps, fixed_tree=False, label="", shapes=None):
    """Runs GPU adt_step and the oracle decoder side by side; returns (steps matched, flag).
    shapes, if a list, receives every compared (d_hat, k_hat)."""
    _, om, dm, pre = _setup(rt, cfg)
    sess = rt.DeviceSession(dm, cfg, fixed_tree=fixed_tree)
    guided = cfg.guidance is not None
    null = synth.null_prefix_ids(cfg) if guided else None
    dec = Decoder(cfg, om, pre, uncond_prefix=null)
    if fixed_tree:
        s = cfg.sched
        dec.schedule_next = lambda: (min(s.d_hi, cfg.n_image - (dec.L + 1 - dec.P) - 1), s.k_hi)
    tol = TOL[cfg.model.dtype]
    g_first = sess.prefill(pre, null)
    o_first = dec.prefill()
    if guided:
        gl = sess.tensors()["logits"][0].cpu().numpy()
        assert _guided_ok(gl, dec.prefill_logits, dec.prefill_branch_logits, cfg.guidance, tol).all(), \
            f"guided prefill logits outside tolerance: {np.abs(gl - dec.prefill_logits).max()}"
    if g_first != o_first:
        return 0, "first token differs (near-tie)"
    matched = 0
    while not dec.done() and matched < n_steps:
        o = dec.step()
        g = sess.step()
        t = sess.tensors()
        print(f"{label} step {o.step}: d={o.d_hat} k={o.k_hat} n={o.tree.n} a={len(o.path)}", flush=True)
        assert (g["d_hat"], g["k_hat"]) == (o.d_hat, o.k_hat), "schedule differs"
        if shapes is not None:
            shapes.append((o.d_hat, o.k_hat))
        if o.draft_root_logits is not None:
            gd = t["draft_logits"][0].cpu().numpy()
            if guided:
                gb = t["draft_branch_logits"].cpu().numpy()
                for b in range(2):
                    assert _tol_ok(gb[b], dec.draft_root_branch_logits[b], tol).all(), \
                        f"draft root logits of branch {b} outside tolerance at step {o.step}"
                ok = _guided_ok(gd, o.draft_root_logits, dec.draft_root_branch_logits, cfg.guidance, tol)
            else:
                ok = _tol_ok(gd, o.draft_root_logits, tol)
            assert ok.all(), \
                f"draft root logits outside tolerance at step {o.step}: {np.abs(gd - o.draft_root_logits).max()}"
        same_tree = (t["n"] == o.tree.n and t["parent"].cpu().tolist() == o.tree.parent.tolist()
                     and t["token"].cpu().tolist() == o.tree.token.tolist())
        if not same_tree:
            return matched, f"tree differs at step {o.step}"
        assert t["depth"].cpu().tolist() == o.tree.depth.tolist()
        glog = t["logits"].cpu().numpy()
        if guided:
            gb = t["branch_logits"].cpu().numpy()
            for b in range(2):
                assert _tol_ok(gb[:, b], dec.verify_branch_logits[b], tol).all(), \
                    f"verify logits of branch {b} outside tolerance at step {o.step}"
            ok = _guided_ok(glog, o.logits, dec.verify_branch_logits, cfg.guidance, tol)
        else:
            ok = _tol_ok(glog, o.logits, tol)
        assert ok.all(), f"verify logits outside tolerance at step {o.step}: max err {np.abs(glog - o.logits).max()}"
        if g["tokens"] != o.committed:
            # near-tie rule: some decision on the oracle's walk had a margin below tolerance
            err = np.abs(glog - o.logits).max()
            walk = [0] + o.path
            margins = [_greedy_margin(o.logits[u], *o.allowed[u]) for u in walk]
            assert min(margins) < 2 * err + tol[0], f"committed tokens differ without a near-tie at step {o.step}"
            return matched, f"near-tie at step {o.step}"
        matched += 1
    return matched, None


def test_tiny_full_image_adt_schedule(rt):
    cfg = synth.get_config("tiny")
    matched, flag = _compare_run(rt, cfg, 10_000, label="tiny")
    print("tiny matched", matched, flag)
    assert flag is None and matched >= 1


INIT_RULES = {"vertical": dict(init="vertical"), "random": dict(init="random", seed=11),
              "tokenflock": dict(init="tokenflock", flock_delta=2), "fixed_d1": dict(fix_d=1),
              "fixed_d1_k3": dict(fix_d=1, fix_k=3), "deep_width": dict(k_clamp="deep", l_k=4)}


@pytest.mark.parametrize("rule", list(INIT_RULES))
def test_tiny_full_image_init_rules(rt, rule):
    """The other initialisation rules (Sec. 4.1, Sec. 5.3 Eqs. 6-8, Table V) and the
    deep-only width bound (Sec. 4.2) through adt_step over a whole image: every schedule
    decision, tree and committed token equal to the oracle's."""
    cfg = synth.get_config("tiny")
    cfg = dataclasses.replace(cfg, sched=dataclasses.replace(cfg.sched, **INIT_RULES[rule]))
    shapes = []
    matched, flag = _compare_run(rt, cfg, 10_000, label="tiny-" + rule, shapes=shapes)
    print(rule, "matched", matched, flag, "shapes", sorted(set(shapes)))
    assert flag is None and matched >= 1
    if rule == "deep_width":
        assert any(k > cfg.sched.k_hi for _, k in shapes)     # one-layer trees wider than k_hi ran
    if rule == "random":
        assert len(set(shapes)) >= 6


@pytest.mark.parametrize("scale,prefix_len", [(3.0, 100), (1.5, 40)])
def test_tiny_full_image_guided(rt, scale, prefix_len):
    """Classifier-free guidance in target and draft (Sec. 3.1, Fig. 5 caption) over the whole
    image: both branches' logits within tolerance, guided logits within the propagated bound,
    schedule, trees and committed tokens bit-exact.  A 100-id prompt is prefilled in two
    chunks (64 nodes = 128 rows, then 36)."""
    cfg = synth.get_config("tiny")
    cfg = dataclasses.replace(cfg, guidance=scale, prefix_len=prefix_len)
    matched, flag = _compare_run(rt, cfg, 10_000, label=f"tiny-guided-{scale}")
    print("guided", scale, "matched", matched, flag)
    assert flag is None and matched >= 1


def test_tiny_fixed_deep_tree(rt):
    cfg = synth.get_config("tiny")
    matched, flag = _compare_run(rt, cfg, 40, fixed_tree=True, label="tiny-fixed")
    print("tiny fixed matched", matched, flag)
    assert flag is None and matched == 40


def _small_bf16():
    cfg = synth.shrink(synth.get_config("llamagen_xl"), n_layers=2, d_model=256, n_heads=4, ffn=512, vocab=512)
    return dataclasses.replace(cfg, prefix_len=16, img_hi=512, prefix_hi=512, grid_h=8, grid_w=8)


def _table_row(depth, token, rows):
    return (depth * 131 + token) % rows


@pytest.mark.parametrize("d_hat,k_hat,n_budget", [(1, 4, 16), (3, 4, 16), (6, 10, 60), (9, 13, 60), (2, 13, 60),
                                                  (4, 1, 60), (5, 7, 127)])
def test_expand_from_table_bit_exact(rt, d_hat, k_hat, n_budget):
    """Expansion and rerank (a2, a3) driven by a caller-supplied draft-logit table: the GPU tree
    must equal the oracle's expansion of the same table (parents, tokens, depths bit-exact,
    scores to fp32 rounding)."""
    from oracle.expand import build_tree, expand
    cfg = synth.get_config("tiny")
    cfg = dataclasses.replace(cfg, sched=dataclasses.replace(cfg.sched, d_hi=9, k_hi=13, n_budget=127))
    _, om, dm, pre = _setup(rt, cfg)
    rows = 97
    table = synth.draw_tensor(77, 5, (rows, cfg.model.vocab), False, std=np.float32(2.0))
    sess = rt.DeviceSession(dm, cfg, draft_table=torch.from_numpy(table).cuda())
    root = sess.prefill(pre)
    n = sess.expand(d_hat, k_hat, n_budget)
    t = sess.tensors()
    tab = table.astype(np.float64)
    L = len(pre)
    level_fn = lambda frontier, pool: np.stack([tab[_table_row(pool[u].depth, pool[u].token, rows)] for u in frontier])
    pool, sel = expand(tab[_table_row(0, root, rows)], level_fn, d_hat, k_hat, n_budget,
                       lambda dp: cfg.allowed(L + dp - len(pre)))
    ref = build_tree(root, pool, sel)
    assert n == ref.n
    assert t["parent"].cpu().tolist() == ref.parent.tolist()
    assert t["token"].cpu().tolist() == ref.token.tolist()
    assert t["depth"].cpu().tolist() == ref.depth.tolist()
    np.testing.assert_allclose(t["score"].cpu().numpy(), ref.score, atol=2e-5, rtol=1e-6)
    from oracle.tree import packed_mask
    assert np.array_equal(t["mask"].cpu().numpy().view(np.uint64), packed_mask(ref.parent, 2))


@pytest.mark.parametrize("d_hat,k_hat,children,n_budget,top_k,T", [(1, 4, 3, 16, 0, 1.0), (3, 4, 3, 16, 0, 1.0),
                                                                    (6, 10, 4, 60, 50, 0.8), (9, 13, 2, 127, 0, 1.3),
                                                                    (4, 2, 16, 60, 0, 1.0)])
def test_expand_sampled_from_table_bit_exact(rt, d_hat, k_hat, children, n_budget, top_k, T):
    """Stochastic children (every expanded node draws its children from q; all drawn children
    kept in creation order; whole expansions within the budget) driven by a caller-supplied
    draft-logit table: the GPU tree equals the oracle's sampled expansion of the same table."""
    from oracle.expand import build_tree, expand_sampled
    cfg = synth.get_config("tiny")
    cfg = dataclasses.replace(cfg, sched=dataclasses.replace(cfg.sched, d_hi=9, k_hi=13, n_budget=127),
                              accept=synth.AcceptCfg(mode="mss", temperature=T, top_k=top_k, children=children))
    _, om, dm, pre = _setup(rt, cfg)
    rows = 97
    table = synth.draw_tensor(78, 5, (rows, cfg.model.vocab), False, std=np.float32(2.0))
    sess = rt.DeviceSession(dm, cfg, draft_table=torch.from_numpy(table).cuda())
    root = sess.prefill(pre)
    n = sess.expand(d_hat, k_hat, n_budget)
    t = sess.tensors()
    tab = table.astype(np.float64)
    L = len(pre)
    level_fn = lambda frontier, pool: np.stack([tab[_table_row(pool[u].depth, pool[u].token, rows)] for u in frontier])
    pool, sel = expand_sampled(tab[_table_row(0, root, rows)], level_fn, d_hat, k_hat, children, n_budget,
                               lambda dp: cfg.allowed(L + dp - len(pre)), temperature=T, top_k=top_k, seed=cfg.seed,
                               step=t["step"])
    ref = build_tree(root, pool, sel, by_creation=True)
    print(f"sampled tree d={d_hat} k={k_hat} c={children}: {ref.n} nodes", flush=True)
    assert n == ref.n
    assert t["parent"].cpu().tolist() == ref.parent.tolist()
    assert t["token"].cpu().tolist() == ref.token.tolist()
    assert t["depth"].cpu().tolist() == ref.depth.tolist()
    np.testing.assert_allclose(t["score"].cpu().numpy(), ref.score, atol=2e-5, rtol=1e-6)


@pytest.mark.parametrize("children,top_k,T", [(3, 0, 1.0), (2, 40, 0.8)])
def test_tiny_cycles_stochastic_children(rt, children, top_k, T):
    """Whole cycles with stochastic children and Eq. 1 as printed (tiny fp32 model, ADT
    schedule): schedule, sampled trees and committed tokens equal the oracle's cycle by
    cycle; every cycle the session's acceptance kernel re-decides the oracle's logits, q rows
    and tree bit for bit (the precision both decide in).  A difference of the sessions' own
    commits is accepted only where that re-decision agrees with the oracle (a draw within the
    fp32 logit error of a boundary); the run then stops."""
    from oracle.accept import accept_mss
    cfg = synth.get_config("tiny")
    cfg = dataclasses.replace(cfg, accept=synth.AcceptCfg(mode="mss", temperature=T, top_k=top_k, children=children))
    _, om, dm, pre = _setup(rt, cfg)
    sess = rt.DeviceSession(dm, cfg)
    dec = Decoder(cfg, om, pre)
    assert sess.prefill(pre) == dec.prefill()
    t_ = lambda x: torch.from_numpy(np.ascontiguousarray(x)).cuda()
    matched = accepted = 0
    while not dec.done() and matched < 60:
        o = dec.step()
        g = sess.step()
        t = sess.tensors()
        assert (g["d_hat"], g["k_hat"]) == (o.d_hat, o.k_hat), f"schedule at step {o.step}"
        assert t["parent"].cpu().tolist() == o.tree.parent.tolist(), f"tree parents at step {o.step}"
        assert t["token"].cpu().tolist() == o.tree.token.tolist(), f"tree tokens at step {o.step}"
        glog = t["logits"].cpu().numpy()
        assert _tol_ok(glog, o.logits, TOL["f32"]).all()
        # the kernel on the oracle's numbers
        n = o.tree.n
        q_nodes = sorted(dec.q_rows)
        q_logits = np.stack([dec.q_rows[u] for u in q_nodes]).astype(np.float32) if q_nodes else \
            np.zeros((1, cfg.model.vocab), np.float32)
        q_row = np.full(n, -1, dtype=np.int32)
        for i, u in enumerate(q_nodes):
            if u < n:
                q_row[u] = i
        tq, tr_ = t_(q_logits), t_(q_row)
        acfg = rt.accept_cfg("mss", T, top_k, seed=cfg.seed, q_logits=tq, q_row=tr_)
        args = [t_(o.logits.astype(np.float32)), t_(o.tree.parent.astype(np.int32)), t_(o.tree.token.astype(np.int32)),
                t_(o.allowed.astype(np.int32)), t_(np.array([n], dtype=np.int32))]
        path, n_acc, bonus = rt.verify_accept(*args, acfg, o.step)
        a = int(n_acc.item())
        assert path[1:a + 1].cpu().tolist() == list(o.path) and int(bonus.item()) == o.bonus, \
            f"shared-number acceptance differs at step {o.step}"
        if g["tokens"] != o.committed:
            print(f"stochastic children: commits differ at step {o.step} (fp32 draw boundary)", flush=True)
            break
        matched += 1
        accepted += len(o.path)
    print(f"stochastic children c={children}: {matched} cycles matched, {accepted} draft tokens accepted", flush=True)
    assert matched >= 30 and accepted > 0


def _planted(rt, cfg, m, extra_rng=0):
    """Planted tree: the oracle's own greedy AR continuation as one chain at random sibling
    ranks plus distractors.  Verify + accept + compact must give a = m, bonus = AR token m+1
    and a compacted cache equal to the oracle's."""
    w, om, dm, pre = _setup(rt, cfg)
    guided = cfg.guidance is not None
    null = synth.null_prefix_ids(cfg) if guided else None
    ar, _ = ar_decode(cfg, om, pre, n_tokens=m + 2, uncond_prefix=null)
    rng = np.random.default_rng(extra_rng)
    V = cfg.model.vocab
    lo, hi = cfg.img_lo, cfg.img_hi
    parent, token = [-1], [ar[0]]
    cur = 0
    for j in range(1, m + 1):
        others = [int(x) for x in rng.choice(np.arange(lo, hi), size=3, replace=False) if int(x) != ar[j]][:2]
        kids = others[: int(rng.integers(0, 3))]
        pos = int(rng.integers(0, len(kids) + 1))
        kids = kids[:pos] + [ar[j]] + kids[pos:]
        base = len(parent)
        for t in kids:
            parent.append(cur)
            token.append(int(t))
        cur = base + kids.index(ar[j])
    # BFS order already holds: each level's children are appended after the previous level
    sess = rt.DeviceSession(dm, cfg)
    first = sess.prefill(pre, null)
    dec = Decoder(cfg, om, pre, uncond_prefix=null)
    assert dec.prefill() == first == ar[0]
    sess.set_tree(parent, token)
    sess.verify()
    t = sess.tensors()
    tree = Tree(np.array(parent, dtype=np.int32), np.array(token, dtype=np.int32), depths(parent),
                np.zeros(len(parent)), np.full(len(parent), -1))
    info = dec.verify_commit(tree, m, 1)
    glog = t["logits"].cpu().numpy()
    tol = TOL[cfg.model.dtype]
    if guided:
        ok = _guided_ok(glog, info.logits, dec.verify_branch_logits, cfg.guidance, tol)
    else:
        ok = _tol_ok(glog, info.logits, tol)
    assert ok.all(), f"max err {np.abs(glog - info.logits).max()}"
    out = sess.accept_commit(m, 1)
    assert out["n_accepted"] == m and out["tokens"] == ar[1:m + 2]
    assert info.committed == out["tokens"]
    L0 = len(pre)
    n_keep = L0 + m + 1
    for b, br in enumerate(dec.branches):
        gk = (sess.k_cache[b] if guided else sess.k_cache).float().cpu().numpy()[:, :, :n_keep]
        gv = (sess.v_cache[b] if guided else sess.v_cache).float().cpu().numpy()[:, :, :n_keep]
        assert _tol_ok(gk, br.tcache.k[:, :, :n_keep], tol).all(), f"compacted K of branch {b}"
        assert _tol_ok(gv, br.tcache.v[:, :, :n_keep], tol).all(), f"compacted V of branch {b}"
    if guided and not dec.done():
        # the next cycle's draft catch-up reads the committed features of both branches
        o, g = dec.step(), sess.step()
        assert (g["d_hat"], g["k_hat"]) == (o.d_hat, o.k_hat)
        gb = sess.tensors()["draft_branch_logits"].cpu().numpy()
        for b in range(2):
            assert _tol_ok(gb[b], dec.draft_root_branch_logits[b], tol).all(), f"draft root of branch {b}"


@pytest.mark.parametrize("m", [0, 1, 3, 4])
def test_planted_path_tiny(rt, m):
    _planted(rt, synth.get_config("tiny"), m, extra_rng=m)


def test_planted_path_bf16_small(rt):
    _planted(rt, _small_bf16(), 5, extra_rng=9)


@pytest.mark.parametrize("m", [0, 3])
def test_planted_path_tiny_guided(rt, m):
    _planted(rt, dataclasses.replace(synth.get_config("tiny"), guidance=3.0), m, extra_rng=m)


def test_planted_path_bf16_small_guided(rt):
    _planted(rt, dataclasses.replace(_small_bf16(), guidance=3.0), 5, extra_rng=9)


@pytest.mark.parametrize("graphs", [(True, True), (True, False)])
def test_determinism(rt, graphs):
    """Two runs are bitwise identical; so are the graph-replayed and the plainly launched path."""
    cfg = _small_bf16()
    outs = []
    for g in graphs:
        _, _, dm, pre = _setup(rt, cfg)
        sess = rt.DeviceSession(dm, cfg, fixed_tree=True, use_graphs=g)
        sess.prefill(pre)
        toks = [sess.step()["tokens"] for _ in range(4)]
        outs.append((toks, sess.tensors()["logits"].cpu().numpy().copy()))
    assert outs[0][0] == outs[1][0] and np.array_equal(outs[0][1], outs[1][1])


# ---------------------------------------------------------------- batched cycle
def _batch_prompts(cfg, B):
    return [synth.prefix_ids(dataclasses.replace(cfg, seed=cfg.seed + 101 * b)) for b in range(B)]


@pytest.mark.parametrize("B,fixed", [(4, False), (5, True), (16, True)])
def test_batch_cycle_matches_single_sessions(rt, B, fixed):
    """adt_batch_step (one verify forward over the packed rows of B trees, MFMA-tiled GEMMs on
    the packed weights, per-sequence attention) against B sessions stepped alone, in lockstep:
    each cycle the single session expands with the batch's (d, k) (root draft logits within
    the bf16 tolerance; its tree equal to the batch's unless the single session's own root
    top-k margin lies inside the observed draft error, or the difference is deeper, where the
    draft inputs already carry the previous verify's rounding), then verifies the batch's tree
    (verify logits within the tolerance) and accepts (committed tokens equal unless the single
    session's argmax margin on the path is inside the observed error; that sequence then
    stops).  The single path itself is checked against the oracle by the tests above.  Fixed
    6-deep, 10-wide trees give 61 rows per tree (M up to 976)."""
    cfg = _small_bf16()
    w, om, dm, _ = _setup(rt, cfg)
    prompts = _batch_prompts(cfg, B)
    batch = rt.DeviceBatch(dm, [cfg] * B, fixed_tree=fixed)
    singles = [rt.DeviceSession(dm, cfg, fixed_tree=fixed, use_graphs=False) for _ in range(B)]
    firsts = batch.prefill(prompts)
    assert firsts == [s.prefill(p) for s, p in zip(singles, prompts)]
    live = [True] * B
    tol = TOL["bf16"]
    stats = {"cycles": 0, "rows": 0, "tree_equal": 0, "tree_level1_ties": 0, "deeper_tree_differs": 0,
             "commit_ties": 0, "oracle_cycles": 0}
    # sequence 0 also against the oracle: its schedule, and its verify of the batch's tree
    dec = Decoder(cfg, om, prompts[0])
    if fixed:
        sc = cfg.sched
        dec.schedule_next = lambda: (min(sc.d_hi, cfg.n_image - (dec.L + 1 - dec.P) - 1), sc.k_hi)
    oracle_live = dec.prefill() == firsts[0]
    for step in range(8):
        outs = batch.step()
        for b in range(B):
            if not live[b]:
                continue
            g, s = outs[b], singles[b]
            if g["n_committed"] == 0:
                live[b] = False
                continue
            d, k = g["d_hat"], g["k_hat"]
            t = batch.sessions[b].tensors()
            bpar, btok = t["parent"].cpu().tolist(), t["token"].cpu().tolist()
            if d >= 1:
                n = s.expand(d, k, cfg.sched.n_budget)
                ts = s.tensors()
                gz, sz = t["draft_logits"][0].cpu().numpy(), ts["draft_logits"][0].cpu().numpy()
                assert _tol_ok(gz, sz, tol).all(), f"sequence {b}: root draft logits"
                if ts["parent"].cpu().tolist() == bpar and ts["token"].cpu().tolist() == btok:
                    stats["tree_equal"] += 1
                else:
                    l1 = lambda par, tok: [tok[i] for i in range(len(par)) if par[i] == 0]
                    if l1(bpar, btok) != l1(ts["parent"].cpu().tolist()[:n], ts["token"].cpu().tolist()[:n]):
                        lo, hi = ts["allowed"].cpu().numpy()[0]
                        z = np.sort(sz[lo:hi].astype(np.float64))[::-1][: k + 1]
                        err = float(np.abs(gz - sz).max())
                        assert np.min(z[:-1] - z[1:]) < 2 * err + tol[0], f"sequence {b}: first level differs"
                        stats["tree_level1_ties"] += 1
                    else:
                        stats["deeper_tree_differs"] += 1
            s.set_tree(bpar, btok)
            s.verify()
            ts = s.tensors()
            glog, slog = t["logits"].cpu().numpy(), ts["logits"].cpu().numpy()
            assert glog.shape == slog.shape
            assert _tol_ok(glog, slog, tol).all(), f"sequence {b}: verify logits max diff {np.abs(glog - slog).max()}"
            if b == 0 and oracle_live and not dec.done():
                assert dec.schedule_next() == (d, k), "schedule differs from the oracle"
                tree = Tree(np.asarray(bpar, np.int32), np.asarray(btok, np.int32), depths(bpar).astype(np.int32),
                            np.zeros(len(bpar)), np.full(len(bpar), -1))
                info = dec.verify_commit(tree, d, k, expanded=d >= 1)
                assert _tol_ok(glog, info.logits, tol).all(), \
                    f"verify logits vs oracle: max diff {np.abs(glog - info.logits).max()}"
                stats["oracle_cycles"] += 1
                if info.committed != g["tokens"]:
                    err = float(np.abs(glog - info.logits).max())
                    margins = [_greedy_margin(info.logits[u], *info.allowed[u]) for u in [0] + info.path]
                    assert min(margins) < 2 * err + tol[0], "tokens differ from the oracle without a near-tie"
                    oracle_live = False
            o = s.accept_commit(d, k)
            stats["cycles"] += 1
            stats["rows"] += len(bpar)
            if g["tokens"] != o["tokens"]:
                err = float(np.abs(glog - slog).max())
                allowed = ts["allowed"].cpu().numpy()
                path = ts["path"].cpu().numpy()[: o["n_accepted"] + 1]
                margins = [_greedy_margin(slog[u], *allowed[u]) for u in path]
                assert min(margins) < 2 * err + tol[0], f"sequence {b}: tokens differ without a near-tie"
                stats["commit_ties"] += 1
                live[b] = False
    print("batch", B, "fixed", fixed, stats)
    assert stats["cycles"] >= B * 6 and stats["oracle_cycles"] >= 4
