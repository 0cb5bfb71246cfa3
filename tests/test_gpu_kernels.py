"""GPU parity of the standalone ABI calls against the oracle, on seeded synthetic inputs.

Floating point: |gpu - oracle| <= atol + rtol * |oracle| with (2e-2, 1e-2) for bf16 and
(1e-5, 1e-5) for fp32.  Integer outputs (masks, depths, paths, tokens, compacted caches)
are compared bit for bit."""
import numpy as np
import pytest
import torch

import synth
from oracle.accept import accept_greedy
from oracle.attention import attend_rows, tree_key_slots
from oracle.decode import compact_cache
from oracle.tree import ancestors_and_self, depths, packed_mask

pytestmark = pytest.mark.gpu

BF16_TOL = (2e-2, 1e-2)
F32_TOL = (1e-5, 1e-5)


def _close(got, ref, tol, what):
    atol, rtol = tol
    err = np.abs(got - ref)
    bad = err > atol + rtol * np.abs(ref)
    assert not bad.any(), f"{what}: {bad.sum()} of {bad.size} outside tolerance, max err {err.max():.3e}"


@pytest.fixture(scope="module")
def rt():
    from paper_2512_21857_amd import runtime
    assert torch.cuda.is_available()
    return runtime


def _dev_tree(rt, parent_np, n_nodes_np):
    parent = torch.from_numpy(parent_np.astype(np.int32)).cuda()
    n = torch.from_numpy(n_nodes_np.astype(np.int32)).cuda()
    mask, dep = rt.tree_masks(parent, n)
    return mask, dep


def _bits_to_f64(b):
    return synth.bf16_bits_to_f32(b).astype(np.float64)


def _attn_case(rt, B, H, Dh, n, l_lo, l_hi, seed, vary_n=False, rows=None):
    ab = synth.attn_microbench(B, H, Dh, n, seed=seed, l_lo=l_lo, l_hi=l_hi, vary_n=vary_n)
    mask, _ = _dev_tree(rt, ab.parent, ab.n_nodes)
    q = torch.from_numpy(ab.q.view(np.int16)).cuda().view(torch.bfloat16)
    k = torch.from_numpy(ab.k.view(np.int16)).cuda().view(torch.bfloat16)
    v = torch.from_numpy(ab.v.view(np.int16)).cuda().view(torch.bfloat16)
    kv_len = torch.from_numpy(ab.kv_len).cuda()
    n_nodes = torch.from_numpy(ab.n_nodes).cuda()
    kv_cap = int((ab.kv_len + ab.n_nodes).max())
    out = rt.tree_attn(q, k, v, kv_len, n_nodes, n_nodes, mask, kv_cap)
    got = out.float().cpu().numpy()
    qf, kf, vf = _bits_to_f64(ab.q), _bits_to_f64(ab.k), _bits_to_f64(ab.v)
    checked = 0
    for b in range(B):
        nb = int(ab.n_nodes[b])
        anc = ancestors_and_self(ab.parent[b, :nb])
        keys = tree_key_slots(int(ab.kv_len[b]), anc)
        sel = range(nb) if rows is None else rows(b, nb)
        for i in sel:
            ref = attend_rows(qf[b, i:i + 1], kf[b], vf[b], [keys[i]], 1.0 / np.sqrt(Dh))[0]
            _close(got[b, i], ref, BF16_TOL, f"tree_attn b={b} i={i}")
            checked += 1
    return checked


@pytest.mark.parametrize("n", [1, 7, 16, 33, 64, 100, 128])
def test_tree_attn_bf16_small(rt, n):
    """Several 64-key tiles and a ragged tail: L in [0, 300]."""
    print(f"tree_attn bf16 n={n}", flush=True)
    assert _attn_case(rt, B=3, H=4, Dh=128, n=n, l_lo=0, l_hi=300, seed=11) == 3 * n


def test_tree_attn_bf16_head64_ragged_batch(rt):
    assert _attn_case(rt, B=5, H=3, Dh=64, n=61, l_lo=1, l_hi=700, seed=12, vary_n=True) > 0


@pytest.mark.parametrize("n", [20, 40, 61])
def test_tree_attn_bf16_long_prefix_split_keys(rt, n):
    """Few (sequence, head) pairs over long prefixes (L in [1500, 2000], head size 128): the keys
    are split across workgroups and merged by the second kernel."""
    print(f"tree_attn bf16 long prefix n={n}", flush=True)
    assert _attn_case(rt, B=2, H=4, Dh=128, n=n, l_lo=1500, l_hi=2000, seed=13) == 2 * n


@pytest.mark.parametrize("B,H,Dh,n,l_lo,l_hi,vary", [
    (8, 16, 64, 40, 0, 300, True),      # shared 64-key blocks, 3 query tiles, keys split in two halves
    (4, 32, 128, 64, 1, 130, False),    # 4 tiles, prefixes shorter than two blocks
    (16, 8, 64, 100, 60, 200, True),    # 7 tiles (one wave only loads), ragged trees
    (2, 64, 128, 128, 0, 70, False),    # 8 tiles, almost no prefix: nearly every block is masked
    (8, 16, 128, 33, 500, 700, False),  # 3 tiles at the smallest row count of that shape
    (8, 16, 128, 32, 100, 400, True),   # 2 tiles at head size 128: four waves, keys split in two halves
    (16, 8, 64, 20, 0, 200, False),     # 2 tiles at head size 64, the smallest tree of the path
    (8, 16, 128, 65, 200, 900, True),   # 5 tiles at head size 128 (three waves only load), ragged trees
    (4, 32, 128, 100, 300, 1100, True), # 7 tiles, prefixes of very different lengths (work-balanced order)
    (8, 16, 128, 96, 0, 150, False),    # 6 tiles over short prefixes: most blocks cross the tree
    (9, 16, 128, 40, 0, 1500, True),    # an odd number of sequences in the work-balanced order
])
def test_tree_attn_bf16_many_pairs_blocks(rt, B, H, Dh, n, l_lo, l_hi, vary):
    """Many (sequence, head) pairs with trees of 17-128 rows take the shared-block kernel."""
    assert _attn_case(rt, B=B, H=H, Dh=Dh, n=n, l_lo=l_lo, l_hi=l_hi, seed=B * 1000 + n, vary_n=vary) > 0


@pytest.mark.parametrize("n", [7, 16])
def test_tree_attn_bf16_many_pairs_one_tile(rt, n):
    """Many (sequence, head) pairs with trees of at most 16 rows at head size 128: one
    workgroup per pair whose waves split the keys (eight waves up to 8 rows, four above),
    ragged trees and prefixes from empty to several hundred keys."""
    print(f"tree_attn bf16 many pairs one tile n={n}", flush=True)
    assert _attn_case(rt, B=8, H=16, Dh=128, n=n, l_lo=0, l_hi=700, seed=8000 + n, vary_n=True) > 0


@pytest.mark.parametrize("n", [5, 16])
def test_tree_attn_bf16_many_pairs_one_tile_head64(rt, n):
    """Many (sequence, head) pairs with trees of at most 16 rows at head size 64: the
    one-workgroup-per-pair kernel with eight waves in the sequence order, ragged trees and
    prefixes from empty to several hundred keys."""
    print(f"tree_attn bf16 many pairs one tile head 64 n={n}", flush=True)
    assert _attn_case(rt, B=16, H=8, Dh=64, n=n, l_lo=0, l_hi=600, seed=9000 + n, vary_n=True) > 0


def test_tree_attn_bf16_full_microbench_sampled(rt):
    """The 16 x 32 x 128 microbenchmark at its real size (L in [512, 2400], 128 nodes), checked
    on sampled rows including the root, the last node and a deep node of every sequence."""
    rows = lambda b, nb: sorted({0, nb - 1, nb // 2, (7 * b + 3) % nb})
    assert _attn_case(rt, B=16, H=32, Dh=128, n=128, l_lo=512, l_hi=2400, seed=3, rows=rows) > 0


def test_tree_attn_f32(rt):
    rng = np.random.default_rng(5)
    B, H, Dh, n = 2, 4, 64, 17
    L = np.array([0, 321], dtype=np.int32)
    S = int(L.max()) + n
    parent = np.stack([synth.random_parents(rng, n) for _ in range(B)])
    q = rng.standard_normal((B, n, H, Dh)).astype(np.float32)
    k = rng.standard_normal((B, H, S, Dh)).astype(np.float32)
    v = rng.standard_normal((B, H, S, Dh)).astype(np.float32)
    nn = np.full(B, n, dtype=np.int32)
    mask, _ = _dev_tree(rt, parent, nn)
    tq, tk, tv = (torch.from_numpy(x).cuda() for x in (q, k, v))
    kvl, nt = torch.from_numpy(L).cuda(), torch.from_numpy(nn).cuda()
    out = rt.tree_attn(tq, tk, tv, kvl, nt, nt, mask, S).cpu().numpy()
    for b in range(B):
        keys = tree_key_slots(int(L[b]), ancestors_and_self(parent[b]))
        ref = attend_rows(q[b].astype(np.float64), k[b].astype(np.float64), v[b].astype(np.float64), keys,
                          1.0 / np.sqrt(Dh))
        _close(out[b], ref, F32_TOL, "tree_attn f32")


def test_tree_masks_bit_exact(rt):
    rng = np.random.default_rng(6)
    B, n_max = 6, 128
    nn = np.array([1, 2, 17, 64, 65, 128], dtype=np.int32)
    parent = np.full((B, n_max), -1, dtype=np.int32)
    for b in range(B):
        parent[b, :nn[b]] = synth.random_parents(rng, int(nn[b]))
    mask, dep = _dev_tree(rt, parent, nn)
    mask = mask.cpu().numpy().view(np.uint64)
    dep = dep.cpu().numpy()
    for b in range(B):
        nb = int(nn[b])
        assert np.array_equal(mask[b, :nb], packed_mask(parent[b, :nb], 2))
        assert np.array_equal(dep[b, :nb], depths(parent[b, :nb]))
        assert not mask[b, nb:].any()


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_kv_compact_bit_exact(rt, dtype):
    rng = np.random.default_rng(7)
    B, slices, Dh = 4, 6, 128
    nn = np.array([2, 13, 40, 128], dtype=np.int32)
    L = np.array([0, 5, 300, 1000], dtype=np.int32)
    S = int((L + nn).max())
    path, a = synth.compaction_paths(rng, nn, a_max=12)
    if dtype == "bf16":
        kb = synth.draw_tensor(9, 1, (B, slices, S, Dh), True, std=np.float32(1.0))
        vb = synth.draw_tensor(9, 2, (B, slices, S, Dh), True, std=np.float32(1.0))
        tk = torch.from_numpy(kb.view(np.int16)).cuda().view(torch.bfloat16)
        tv = torch.from_numpy(vb.view(np.int16)).cuda().view(torch.bfloat16)
        rk, rv = kb.copy(), vb.copy()
    else:
        rk = rng.standard_normal((B, slices, S, Dh)).astype(np.float32)
        rv = rng.standard_normal((B, slices, S, Dh)).astype(np.float32)
        tk, tv = torch.from_numpy(rk.copy()).cuda(), torch.from_numpy(rv.copy()).cuda()
    rt.kv_compact(tk, tv, torch.from_numpy(L).cuda(), torch.from_numpy(path).cuda(), torch.from_numpy(a).cuda(),
                  int(a.max()))
    for b in range(B):
        compact_cache(rk[b], rv[b], int(L[b]), [int(x) for x in path[b, 1:a[b] + 1]])
    gk = tk.view(torch.int16).cpu().numpy().view(np.uint16) if dtype == "bf16" else tk.cpu().numpy()
    gv = tv.view(torch.int16).cpu().numpy().view(np.uint16) if dtype == "bf16" else tv.cpu().numpy()
    assert np.array_equal(gk, rk) and np.array_equal(gv, rv)


def test_accept_greedy_planted(rt):
    """Trees holding a planted chain of length m at random sibling ranks: the GPU walk must
    return exactly the oracle's path and bonus."""
    rng = np.random.default_rng(8)
    V = 1000
    for trial in range(30):
        m = int(rng.integers(0, 8))
        n = int(rng.integers(m + 1, 61))
        parent = synth.random_parents(rng, n, max_children=4, max_depth=12)
        token = rng.integers(0, V, size=n).astype(np.int32)
        for u in range(n):                        # siblings carry distinct tokens
            kids = [c for c in range(n) if parent[c] == u]
            token[kids] = rng.choice(V, size=len(kids), replace=False)
        logits = rng.standard_normal((n, V)).astype(np.float32)
        u = 0
        for _ in range(m):
            kids = [c for c in range(n) if parent[c] == u]
            if not kids:
                break
            c = int(rng.choice(kids))
            logits[u, token[c]] = 9.0
            u = c
        lo = int(rng.integers(0, 50))
        allowed = np.tile([lo, V], (n, 1)).astype(np.int32)
        ref_path, ref_bonus = accept_greedy(logits.astype(np.float64), parent, token, allowed)
        cfg = rt.accept_cfg("greedy")
        t = lambda x: torch.from_numpy(np.ascontiguousarray(x)).cuda()
        path, n_acc, bonus = rt.verify_accept(t(logits), t(parent.astype(np.int32)), t(token), t(allowed),
                                              t(np.array([n], dtype=np.int32)), cfg, 0)
        a = int(n_acc.item())
        assert a == len(ref_path) and path[1:a + 1].cpu().tolist() == ref_path and int(bonus.item()) == ref_bonus


def _random_tree_tokens(rng, n, V, lo, hi):
    parent = synth.random_parents(rng, n, max_children=6, max_depth=9)
    token = np.zeros(n, dtype=np.int32)
    for u in range(n):
        kids = [c for c in range(n) if parent[c] == u]
        token[kids] = rng.choice(np.arange(lo, hi), size=len(kids), replace=False)
    return parent.astype(np.int32), token


@pytest.mark.parametrize("mode,top_k,T,ties", [("exact", 2000, 1.0, False), ("exact", 0, 0.7, False),
                                               ("exact", 3, 1.0, False), ("relaxed", 2000, 1.0, False),
                                               ("relaxed", 50, 1.3, False), ("exact", 2000, 1.0, True),
                                               ("relaxed", 700, 1.0, True)])
def test_accept_sampling_bit_exact(rt, mode, top_k, T, ties):
    """Exact / relaxed acceptance on the same fp32 logits: identical path and bonus for every
    (seed, step).  Logits are sharpened on planted chains so long paths get accepted too.
    ties: the logits lie on a grid of 0.5, so hundreds of ids share the value at the top-k
    boundary and the lower ids among them are the ones kept."""
    from oracle.accept import accept_sampling
    rng = np.random.default_rng(21)
    V, lo, hi = 8448, 0, 8192
    knn = synth.random_knn_table(hi, 100, seed=4)
    tk = torch.from_numpy(knn).cuda()
    t = lambda x: torch.from_numpy(np.ascontiguousarray(x)).cuda()
    agree = total_acc = 0
    for trial in range(24):
        n = int(rng.integers(1, 62))
        parent, token = _random_tree_tokens(rng, n, V, lo, hi)
        logits = (rng.standard_normal((n, V)) * 1.5).astype(np.float32)
        if ties:
            logits = np.round(logits * 2.0) / 2.0
        for u in range(n):
            kids = [c for c in range(n) if parent[c] == u]
            if kids and rng.random() < 0.7:
                logits[u, token[kids[0]]] += 7.0
        allowed = np.tile([lo, hi], (n, 1)).astype(np.int32)
        for step in range(3):
            seed = 1000 + trial
            kw = dict(temperature=T, top_k=top_k, seed=seed, step=step, mode=mode)
            if mode == "relaxed":
                kw.update(delta=0.1, knn=knn, knn_k=100)
            ref_path, ref_bonus = accept_sampling(logits, parent, token, allowed, **kw)
            cfg = rt.accept_cfg(mode, T, top_k, 0.1 if mode == "relaxed" else 0.0, tk if mode == "relaxed" else None,
                                100 if mode == "relaxed" else 1, seed)
            path, n_acc, bonus = rt.verify_accept(t(logits), t(parent), t(token), t(allowed),
                                                  t(np.array([n], dtype=np.int32)), cfg, step)
            a = int(n_acc.item())
            assert path[1:a + 1].cpu().tolist() == ref_path and int(bonus.item()) == ref_bonus, \
                f"trial {trial} step {step}"
            agree += 1
            total_acc += a
    assert agree == 72 and total_acc > 0


@pytest.mark.parametrize("top_k,T", [(0, 1.0), (2000, 1.0), (3, 0.7), (50, 1.3)])
def test_accept_mss_bit_exact(rt, top_k, T):
    """Eq. 1 as printed with stochastic children (min(1, p/q), residual norm(max(0, p - q)) in
    128-bit integer arithmetic): identical path and bonus to the oracle for every (seed, step)
    on the same fp32 target and draft rows.  q rows are p rows plus noise, so p/q is near 1
    and long paths are accepted; some nodes get an unrelated q (many rejections, residuals)."""
    from oracle.accept import accept_mss
    rng = np.random.default_rng(31)
    V, lo, hi = 8448, 0, 8192
    t = lambda x: torch.from_numpy(np.ascontiguousarray(x)).cuda()
    agree = total_acc = rejections = 0
    for trial in range(16):
        n = int(rng.integers(1, 62))
        parent, token = _random_tree_tokens(rng, n, V, lo, hi)
        logits = (rng.standard_normal((n, V)) * 1.5).astype(np.float32)
        q_logits = np.zeros((n + 1, V), dtype=np.float32)
        q_row = np.full(n, -1, dtype=np.int32)
        for u in range(n):
            kids = [c for c in range(n) if parent[c] == u]
            if not kids:
                continue
            q_row[u] = u + 1
            if rng.random() < 0.75:
                q_logits[u + 1] = logits[u] + (rng.standard_normal(V) * 0.3).astype(np.float32)
                logits[u, token[kids[0]]] += 8.0
                q_logits[u + 1, token[kids[0]]] += 8.0
            else:
                q_logits[u + 1] = (rng.standard_normal(V) * 1.5).astype(np.float32)
        allowed = np.tile([lo, hi], (n, 1)).astype(np.int32)
        q_map = {u: q_logits[q_row[u]] for u in range(n) if q_row[u] >= 0}
        tq, tr = t(q_logits), t(q_row)
        for step in range(3):
            seed = 2000 + trial
            ref_path, ref_bonus = accept_mss(logits, q_map, parent, token, allowed, temperature=T, top_k=top_k,
                                             seed=seed, step=step)
            cfg = rt.accept_cfg("mss", T, top_k, seed=seed, q_logits=tq, q_row=tr)
            path, n_acc, bonus = rt.verify_accept(t(logits), t(parent), t(token), t(allowed),
                                                  t(np.array([n], dtype=np.int32)), cfg, step)
            a = int(n_acc.item())
            assert path[1:a + 1].cpu().tolist() == ref_path and int(bonus.item()) == ref_bonus, \
                f"trial {trial} step {step}"
            agree += 1
            total_acc += a
            u = ref_path[-1] if ref_path else 0
            rejections += any(parent[c] == u for c in range(n))
    assert agree == 48 and total_acc > 20 and rejections >= 3


def test_accept_sampling_law_on_gpu(rt):
    """Committed first token over 4000 steps on the GPU follows p (chi-square), root with 3 children."""
    V = 16
    rng = np.random.default_rng(3)
    root = rng.standard_normal(V).astype(np.float32)
    parent = np.array([-1, 0, 0, 0], dtype=np.int32)
    token = np.array([0, 5, 2, 9], dtype=np.int32)
    logits = np.vstack([root, rng.standard_normal((3, V)).astype(np.float32)])
    allowed = np.tile([0, V], (4, 1)).astype(np.int32)
    t = lambda x: torch.from_numpy(np.ascontiguousarray(x)).cuda()
    tl, tp, tt, ta, tn = t(logits), t(parent), t(token), t(allowed), t(np.array([4], dtype=np.int32))
    cfg = rt.accept_cfg("exact", 1.0, 0, 0.0, None, 1, 77)
    trials = 4000
    counts = np.zeros(V)
    for s in range(trials):
        path, n_acc, bonus = rt.verify_accept(tl, tp, tt, ta, tn, cfg, s)
        a = int(n_acc.item())
        counts[token[int(path[1].item())] if a > 0 else int(bonus.item())] += 1
    p = np.exp(root.astype(np.float64) - root.max())
    p /= p.sum()
    chi2 = float(np.sum((counts - trials * p) ** 2 / (trials * p)))
    assert chi2 < 45.0          # 15 dof


def _gemm_ref_check(got, x, w, rows):
    """got[rows] against the fp64 product of the bf16 inputs, within the fp32 accumulation bound
    2 K eps sum|x_k w_k| per element (eps = 2^-24)."""
    xf, wf = x[rows].astype(np.float64), w.astype(np.float64)
    ref = xf @ wf.T
    bound = 2.0 * x.shape[1] * 2.0 ** -24 * (np.abs(xf) @ np.abs(wf).T) + 1e-30
    err = np.abs(got[rows] - ref)
    assert (err <= bound).all(), f"max err {err.max()} (bound there {bound.flat[err.argmax()]})"


@pytest.mark.parametrize("M,N,K", [(1, 128, 64), (100, 256, 128), (300, 512, 192), (250, 32768, 128),
                                   (200, 65536, 64)])
def test_gemm_bf16_batched(rt, M, N, K):
    """All three tile shapes (128x128, 256x128, 256x256) and partial row blocks, every element."""
    print(f"gemm_bf16 M={M} N={N} K={K}", flush=True)
    rng = np.random.default_rng(M + N + K)
    xb = rng.standard_normal((M, K)).astype(np.float32)
    wb = rng.standard_normal((N, K)).astype(np.float32)
    xt = torch.from_numpy(xb).cuda().bfloat16()
    wt = torch.from_numpy(wb).cuda().bfloat16()
    got = rt.gemm_bf16(xt, wt).cpu().numpy()
    _gemm_ref_check(got, xt.float().cpu().numpy(), wt.float().cpu().numpy(), np.arange(M))


@pytest.mark.parametrize("M,N,K", [(300, 32768, 128), (1, 65536, 64), (100, 256, 128), (520, 16384, 192),
                                   (300, 512, 8192), (40, 1024, 8256), (130, 384, 320), (976, 3840, 1280),
                                   (976, 12288, 512), (300, 35840, 512), (976, 22016, 320), (500, 1280, 2048)])
def test_gemm_bf16_packed(rt, M, N, K):
    """Packed weights: the DMA pipeline in 256 x 256 blocks (>= 128 of them; K below and above
    the stages it keeps in flight; one row; partial row blocks), with K split over 4
    workgroups per block (few blocks, long K; uneven ranges at K = 8256), and in 128 x 128
    blocks of four waves (few blocks, short K: the narrow projections of a batch of trees),
    in 384 x 128 blocks (976 x 12288: 256 of them against 192 of 256 x 256), and with a last
    round of blocks at most half full moved to a second launch with K split (35840 columns
    over 2 row blocks: 256 + 24 blocks, the 24 split four ways; 22016 over 4: 256 + 88, split
    two ways), every element.  Without a K split the result
    equals the row-major kernel bit for bit (same summation order); the split result is
    checked against the bound and, with the workspace withheld, the unsplit result is the
    row-major one again."""
    print(f"gemm_bf16_packed M={M} N={N} K={K}", flush=True)
    rng = np.random.default_rng(M * 7 + N + K)
    xt = torch.from_numpy(rng.standard_normal((M, K)).astype(np.float32)).cuda().bfloat16()
    wt = torch.from_numpy(rng.standard_normal((N, K)).astype(np.float32)).cuda().bfloat16()
    wp = rt.pack_bf16(wt)
    got = rt.gemm_bf16_packed(xt, wp, N)
    _gemm_ref_check(got.cpu().numpy(), xt.float().cpu().numpy(), wt.float().cpu().numpy(), np.arange(M))
    split = rt.lib().adt_gemm_bf16_packed_workspace_size(M, N, K) > 0
    # 500 x 1280 x 2048: 40 blocks of 128 x 128 with K >= 2048, K split in two
    assert split == (K >= 8192 or N in (35840, 22016) or (M, N, K) == (500, 1280, 2048))
    ref = rt.gemm_bf16(xt, wt)
    if split:
        assert torch.equal(rt.gemm_bf16_packed(xt, wp, N, split=False), ref)
        assert torch.equal(rt.gemm_bf16_packed(xt, wp, N), got)   # deterministic
    else:
        assert torch.equal(got, ref)


def test_gemm_bf16_packed_verify_shapes_sampled(rt):
    """M = 976 (16 trees of 61 rows) with the 7B-shaped projections the benchmark times, on
    sampled rows: QKV 4096 x 12288 and the LM head 4096 x 65536 (DMA pipeline, 256 x 256), O
    4096 x 4096 (128 x 128) and down 11008 x 4096 (256 x 256 with K split in four)."""
    rng = np.random.default_rng(977)
    rows = np.array([0, 1, 31, 32, 255, 256, 511, 767, 768, 900, 975])
    for K, N in ((4096, 12288), (4096, 65536), (4096, 4096), (11008, 4096)):
        print(f"gemm_bf16_packed M=976 N={N} K={K}", flush=True)
        xt = torch.from_numpy(rng.standard_normal((976, K)).astype(np.float32)).cuda().bfloat16()
        wt = torch.from_numpy(rng.standard_normal((N, K)).astype(np.float32)).cuda().bfloat16()
        got = rt.gemm_bf16_packed(xt, rt.pack_bf16(wt), N)
        xs, ws = xt.float().cpu().numpy(), wt.float().cpu().numpy()
        _gemm_ref_check(got.cpu().numpy(), xs, ws, rows)
        if rt.lib().adt_gemm_bf16_packed_workspace_size(976, N, K) == 0:
            assert torch.equal(got, rt.gemm_bf16(xt, wt))
        del xt, wt, got
        torch.cuda.empty_cache()


def test_gemm_bf16_batched_verify_shape_sampled(rt):
    """M = 976 (16 trees of 61 rows) against a 4096 x 4096 projection, on sampled rows."""
    rng = np.random.default_rng(976)
    xt = torch.from_numpy(rng.standard_normal((976, 4096)).astype(np.float32)).cuda().bfloat16()
    wt = torch.from_numpy(rng.standard_normal((4096, 4096)).astype(np.float32)).cuda().bfloat16()
    got = rt.gemm_bf16(xt, wt).cpu().numpy()
    rows = np.array([0, 1, 31, 32, 255, 256, 511, 767, 768, 900, 975])
    _gemm_ref_check(got, xt.float().cpu().numpy(), wt.float().cpu().numpy(), rows)


def test_sample_weights_match_oracle(rt):
    """The device's sampling weights w = rint(exp(d) 2^32) against the oracle's definition of
    the same fixed double sequence, bit for bit: every float32 exponent on a dense grid of
    [-45, 0], random ones, and the edges (0, -0, the -40 cut and its neighbours, -inf)."""
    from oracle.accept import quantised_exp_weight
    rng = np.random.default_rng(14)
    edge = np.array([0.0, -0.0, -40.0, np.nextafter(np.float32(-40.0), np.float32(0.0)),
                     np.nextafter(np.float32(-40.0), np.float32(-50.0)), -1e-30, -np.inf], dtype=np.float32)
    d = np.concatenate([(-np.linspace(0.0, 45.0, 2_000_001)).astype(np.float32),
                        (-rng.random(1_000_000) * 45.0).astype(np.float32), edge])
    dd = torch.from_numpy(d).cuda()
    w = torch.empty(d.size, dtype=torch.int64, device="cuda")
    rt.check(rt.lib().adt_probe_sample_weights(rt._p(dd), d.size, rt._p(w), rt._stream()))
    torch.cuda.synchronize()
    got = w.cpu().numpy()
    ref = quantised_exp_weight(d).astype(np.int64)
    bad = np.flatnonzero(got != ref)
    assert bad.size == 0, f"{bad.size} weights differ, first at d = {d[bad[:4]]}: {got[bad[:4]]} vs {ref[bad[:4]]}"
