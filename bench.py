#!/usr/bin/env python3
"""Throughput of the ADT-Tree draft-then-verify cycle on one MI355X.

A step is one adt_step call: ADT schedule, draft-tree expansion (draft forwards, top-k,
scoring, rerank), the tree-masked verification forward of the target model, greedy
acceptance, KV compaction and commit.  The workload is the LlamaGen-XL-shaped synthetic
model (36 layers, d_model 1280, 20 x 64 heads, SwiGLU 3584, vocab 16384, bf16, seeded
N(0, 0.02) weights), a 120-token seeded prompt and a 32 x 32 image grid, trees of at most
60 draft nodes, width <= 10, depth <= 6.  The metric is verified draft-tree nodes per
second; the line also carries the roofline of the dominant kernel (the weight-streaming
projections), tree-attention bandwidth (in the cycle and in the 16 x 32 x 128 tree-attention
microbenchmark), the batched verify projections, the same cycle under classifier-free
guidance (scale 3.0: both branches in every forward), 16 images decoded together (one verify
forward over all their trees per step), the cycle with stochastic children (drawn from q,
verified by Eq. 1 as printed) and the CPU oracle timed on this host.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

HBM_PEAK_GBS = 8000.0
ROOT = os.path.dirname(os.path.abspath(__file__))
# the sources the GEMM kernel is compiled from (kernel, shared helpers, epilogue struct)
GEMM_SRCS = [os.path.join(ROOT, "paper_2512_21857_amd", "csrc", *parts)
             for parts in (("kernels", "gemm.hip"), ("common.h",), ("launch.h",))]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "gemm_tile_llamagen_xl_traffic.md")


def gemm_traffic():
    """HBM bytes per GEMM launch from the committed FETCH_SIZE / WRITE_SIZE counter summary,
    or None when the kernel's sources changed since the counters were taken (sha256 over
    gemm.hip, common.h and launch.h, in that order)."""
    import hashlib
    try:
        text = open(TRAFFIC_FILE).read()
        h = hashlib.sha256()
        for path in GEMM_SRCS:
            h.update(open(path, "rb").read())
        src = h.hexdigest()
    except OSError:
        return None
    keys = ("source_sha256:", "traffic_bytes_per_launch:")
    fields = dict(line.split(":", 1) for line in text.splitlines() if line.startswith(keys))
    if fields.get("source_sha256", "").strip() != src:
        return None
    return int(fields["traffic_bytes_per_launch"].strip())


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--profile-steps", type=int, default=30)
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--no-microbench", action="store_true")
    ap.add_argument("--no-fixed", action="store_true")
    ap.add_argument("--no-mfma", action="store_true")
    ap.add_argument("--no-guided", action="store_true")
    ap.add_argument("--no-batch", action="store_true")
    ap.add_argument("--no-stochastic", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="first copy 512 MiB device-to-device (a kernel of known traffic for counter scaling)")
    return ap.parse_args()


def run_steps(sess, k):
    import torch
    nodes = tokens = depth = 0
    for _ in range(k):
        o = sess.step()
        nodes += o["n_nodes"] - 1
        tokens += o["n_committed"]
        depth += o["d_hat"]
    torch.cuda.synchronize()
    return nodes, tokens, depth


def timed(sess, k):
    import torch
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    nodes, tokens, depth = run_steps(sess, k)
    torch.cuda.synchronize()
    return time.perf_counter() - t0, nodes, tokens, depth


def profile_pass(rt, abi, sess, k):
    """Per-kernel-class HIP-event timing over k further steps of the same session."""
    import ctypes as C
    L = abi.lib()
    abi.check(L.adt_profile_enable(1))
    for cls in (abi.PROF_GEMM, abi.PROF_ATTN, abi.PROF_COMPACT):
        L.adt_profile_read(cls, None, None, None, None, 1)
    run_steps(sess, k)
    out = {}
    for name, cls in (("gemm", abi.PROF_GEMM), ("attn", abi.PROF_ATTN), ("compact", abi.PROF_COMPACT)):
        n, ms, by, fl = C.c_int64(), C.c_double(), C.c_double(), C.c_double()
        abi.check(L.adt_profile_read(cls, C.byref(n), C.byref(ms), C.byref(by), C.byref(fl), 1))
        out[name] = {"launches": n.value, "ms": ms.value, "bytes": by.value, "flops": fl.value}
    abi.check(L.adt_profile_enable(0))
    return out


def attn_microbench(rt, sizes=(8, 16, 32, 64, 128), iters=30, sets=3):
    """Tree attention alone at 16 sequences x 32 heads x 128, KV length U[512, 2400]; several
    cache sets rotate so the 256 MB last-level cache cannot hold the working set."""
    import torch
    import synth
    out = {}
    for n in sizes:
        bufs = []
        for s in range(sets):
            ab = synth.attn_microbench(16, 32, 128, n, seed=3 + 100 * s)
            dev = lambda a: torch.from_numpy(a.view(np.int16)).cuda().view(torch.bfloat16)
            parent = torch.from_numpy(ab.parent).cuda()
            nn = torch.from_numpy(ab.n_nodes).cuda()
            mask, _ = rt.tree_masks(parent, nn)
            kv_cap = int((ab.kv_len + ab.n_nodes).max())
            bufs.append((dev(ab.q), dev(ab.k), dev(ab.v), torch.from_numpy(ab.kv_len).cuda(), nn, mask, kv_cap,
                         int(ab.kv_len.sum()), int(ab.n_nodes.sum())))
        ws = torch.empty(2 * rt.lib().adt_tree_attn_workspace_size(16, 32, 128, n, 4096) + 256, dtype=torch.uint8,
                         device="cuda")
        outs = [torch.empty_like(b[0]) for b in bufs]
        for i in range(10):
            b = bufs[i % sets]
            rt.tree_attn(b[0], b[1], b[2], b[3], b[4], b[4], b[5], b[6], out=outs[i % sets], workspace=ws)
        st = torch.cuda.current_stream()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(st)
        byts = 0.0
        for i in range(iters):
            b = bufs[i % sets]
            rt.tree_attn(b[0], b[1], b[2], b[3], b[4], b[4], b[5], b[6], out=outs[i % sets], workspace=ws)
            H, Dh = 32, 128
            byts += 2.0 * b[7] * H * Dh * 2 + 4.0 * b[8] * H * Dh * 2 + 16.0 * b[8]
        e1.record(st)
        e1.synchronize()
        ms = e0.elapsed_time(e1) / iters
        gbs = byts / iters / (ms * 1e-3) / 1e9
        out[str(n)] = {"us": round(ms * 1e3, 2), "GB_s": round(gbs, 1), "frac": round(gbs / HBM_PEAK_GBS, 4)}
        del bufs, outs
        torch.cuda.empty_cache()
    return out


def compact_microbench(rt, B=16, layers=36, heads=20, Dh=64, a=6, nodes=61, iters=30):
    """KV compaction alone at the LlamaGen-XL cache shape (16 sequences x 36 layers x 20
    heads, head size 64, bf16), every sequence committing a = 6 accepted nodes of a 61-node
    tree (path[m] an increasing draw from the tree's slots).  Call i moves its rows at prefix
    lengths shifted by i trees, so the rows it touches are not in the last-level cache."""
    import torch
    slices, step = layers * heads, nodes + 8
    rng = np.random.default_rng(17)
    base = rng.integers(256, 513, size=B)
    S_cap = int(base.max()) + step * (iters + 3) + nodes
    gen = torch.Generator(device="cuda")
    gen.manual_seed(17)
    k = torch.randn((B, slices, S_cap, Dh), generator=gen, device="cuda", dtype=torch.bfloat16)
    v = torch.randn((B, slices, S_cap, Dh), generator=gen, device="cuda", dtype=torch.bfloat16)
    path = np.zeros((B, a + 1), np.int32)
    for b in range(B):
        path[b, 1:] = np.sort(rng.choice(np.arange(1, nodes), size=a, replace=False))
    path_t = torch.from_numpy(path).cuda()
    n_acc = torch.full((B,), a, dtype=torch.int32, device="cuda")
    lens = [torch.from_numpy((base + step * i).astype(np.int32)).cuda() for i in range(iters + 3)]
    for i in range(3):
        rt.kv_compact(k, v, lens[iters + i], path_t, n_acc, a)
    st = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(st)
    for i in range(iters):
        rt.kv_compact(k, v, lens[i], path_t, n_acc, a)
    e1.record(st)
    e1.synchronize()
    ms = e0.elapsed_time(e1) / iters
    byts = 2.0 * 2 * B * slices * a * Dh * 2   # K and V rows, each read once and written once
    gbs = byts / (ms * 1e-3) / 1e9
    del k, v
    torch.cuda.empty_cache()
    return {"us": round(ms * 1e3, 2), "GB_s": round(gbs, 1), "frac": round(gbs / HBM_PEAK_GBS, 4),
            "bytes": int(byts), "workload": f"{B} sequences x {layers} layers x {heads} heads x {Dh}, "
            f"{a} accepted nodes of {nodes} per sequence, bf16"}


MFMA_PEAK_TFLOPS = 2500.0
BATCHED_SHAPES = ((4096, 12288), (4096, 4096), (4096, 22016), (11008, 4096), (4096, 65536))


def mfma_benchmark(rt, M=976, iters=10):
    """The verify projections of 16 trees of 61 rows at once (M = 976) with the 7B-shaped
    layer dimensions (K, N): QKV, O, gate/up, down, LM head, weights in the library's packed
    layout (as every model weight is kept).  MFMA-bound (AI >> 315 flop/B).  The vendor BLAS
    (torch.mm, bf16 out) on the same operands is timed beside it for context."""
    import torch
    torch.manual_seed(5)
    out, tot_fl, tot_ms, tot_ref = {}, 0.0, 0.0, 0.0

    def ev_time(f):
        for _ in range(2):
            f()
        st = torch.cuda.current_stream()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(st)
        for _ in range(iters):
            f()
        e1.record(st)
        e1.synchronize()
        return e0.elapsed_time(e1) / iters

    for K, N in BATCHED_SHAPES:
        x = torch.randn(M, K, device="cuda").bfloat16()
        w = torch.randn(N, K, device="cuda").bfloat16()
        wp = rt.pack_bf16(w)
        c = torch.empty(M, N, dtype=torch.float32, device="cuda")
        ms = ev_time(lambda: rt.gemm_bf16_packed(x, wp, N, out=c))
        cb = torch.empty(M, N, dtype=torch.bfloat16, device="cuda")
        wt = w.t()
        ref_ms = ev_time(lambda: torch.mm(x, wt, out=cb))
        fl = 2.0 * M * N * K
        tot_fl += fl
        tot_ms += ms
        tot_ref += ref_ms
        out[f"{K}x{N}"] = {"us": round(ms * 1e3, 1), "TFLOP_s": round(fl / ms / 1e9, 1),
                           "vendor_blas_TFLOP_s": round(fl / ref_ms / 1e9, 1)}
        del x, w, wp, c, cb, wt
    torch.cuda.empty_cache()
    tf = tot_fl / tot_ms / 1e9
    ref_tf = tot_fl / tot_ref / 1e9
    return {"M": M, "shapes_KxN": out, "total_us": round(tot_ms * 1e3, 1), "TFLOP_s": round(tf, 1),
            "peak_TFLOP_s": MFMA_PEAK_TFLOPS, "frac": round(tf / MFMA_PEAK_TFLOPS, 4),
            "vendor_blas": {"TFLOP_s": round(ref_tf, 1), "frac": round(ref_tf / MFMA_PEAK_TFLOPS, 4),
                            "call": "torch.mm bf16 -> bf16 (hipBLASLt), same operands"},
            "kernel": "gemm_nt_dma_kernel (>= 128 blocks of 256x256: global->LDS DMA ring) / gemm_nt_kernel "
                      "(bf16 MFMA 32x32x16, fp32 out)"}


def cpu_baseline(cfg, weights, budget_s):
    """The oracle as it stands, on this host's cores, over the first cycles of the same
    workload (prefill untimed, then as many cycles as fit in the budget)."""
    import threadpoolctl  # noqa: F401
    from oracle.decode import Decoder
    from oracle.model import OracleModel
    import synth
    cores = len(os.sched_getaffinity(0))
    om = OracleModel(cfg, weights)
    dec = Decoder(cfg, om, synth.prefix_ids(cfg))
    dec.prefill()
    nodes = steps = 0
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < budget_s and not dec.done():
        info = dec.step()
        nodes += info.tree.n - 1
        steps += 1
    dt = time.perf_counter() - t0
    try:
        from threadpoolctl import threadpool_info
        blas = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        blas = cores
    return {"value": round(nodes / dt, 3), "unit": "nodes/s", "cores": int(min(cores, blas)), "kind": "oracle",
            "sample": f"fp64 NumPy oracle, prefill untimed then {steps} ADT cycles ({nodes} draft nodes) of the "
                      f"same workload in {dt:.1f} s"}


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; use --gpus 1"}))
        sys.exit(2)
    import torch
    sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
    import synth
    from paper_2512_21857_amd import abi, runtime as rt
    if not torch.cuda.is_available():
        raise SystemExit("bench.py needs a GPU")
    if args.copy_calibration:
        src = torch.ones(128 * 1024 * 1024, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    cfg = synth.get_config("llamagen_xl")
    print(f"[bench] generating weights for {cfg.name}", file=sys.stderr, flush=True)
    w = synth.model_weights(cfg, threads=min(16, os.cpu_count() or 8))
    dm = rt.DeviceModel(cfg, w)
    pre = synth.prefix_ids(cfg)

    def fresh(fixed=False):
        s = rt.DeviceSession(dm, cfg, fixed_tree=fixed)
        s.prefill(pre)
        return s

    def guided_run(k):
        """The same cycle with classifier-free guidance (scale 3.0, conditional and
        unconditional branches in every forward)."""
        import dataclasses
        gcfg = dataclasses.replace(cfg, guidance=3.0)
        gs = rt.DeviceSession(dm, gcfg)
        gs.prefill(pre, synth.null_prefix_ids(gcfg))
        run_steps(gs, 3)
        gdt, gnodes, gtokens, gdepth = timed(gs, k)
        del gs
        return {"scale": 3.0, "nodes_per_s": round(gnodes / gdt, 2), "ms_per_step": round(gdt / k * 1e3, 4),
                "nodes_per_step": round(gnodes / k, 2), "tokens_per_step": round(gtokens / k, 3),
                "mean_depth": round(gdepth / k, 3), "steps": k}

    def stochastic_run(k, children=3):
        """The same cycle with stochastic children (children drawn from q at T = 1, every drawn
        child kept, Eq. 1 acceptance with the residual norm(max(0, p - q)))."""
        import dataclasses
        scfg = dataclasses.replace(cfg, accept=synth.AcceptCfg(mode="mss", temperature=1.0, top_k=0,
                                                                children=children))
        ss = rt.DeviceSession(dm, scfg)
        ss.prefill(pre)
        run_steps(ss, 3)
        sdt, snodes, stokens, sdepth = timed(ss, k)
        del ss
        return {"children": children, "temperature": 1.0, "nodes_per_s": round(snodes / sdt, 2),
                "ms_per_step": round(sdt / k * 1e3, 4), "nodes_per_step": round(snodes / k, 2),
                "tokens_per_step": round(stokens / k, 3), "mean_depth": round(sdepth / k, 3), "steps": k}

    def batched_run(B, fixed, k):
        """B images decoded together: per image its own schedule and draft tree, one verify
        forward over the packed rows of all B trees per step (packed-weight MFMA GEMMs)."""
        import dataclasses
        prompts = [synth.prefix_ids(dataclasses.replace(cfg, seed=cfg.seed + 101 * b)) for b in range(B)]
        bt = rt.DeviceBatch(dm, [cfg] * B, fixed_tree=fixed)
        bt.prefill(prompts)

        def go(n):
            nodes = tokens = 0
            for _ in range(n):
                for o in bt.step():
                    nodes += max(o["n_nodes"] - 1, 0)
                    tokens += o["n_committed"]
            torch.cuda.synchronize()
            return nodes, tokens
        go(3)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        nodes, tokens = go(k)
        bdt = time.perf_counter() - t0
        del bt
        torch.cuda.empty_cache()
        return {"batch": B, "tree": "depth 6, width 10, top-60" if fixed else "ADT schedule per image",
                "nodes_per_s": round(nodes / bdt, 2), "ms_per_step": round(bdt / k * 1e3, 4),
                "rows_per_step": round((nodes + B * k) / k, 1), "tokens_per_step": round(tokens / k, 3),
                "steps": k}

    sess = fresh()
    run_steps(sess, args.warmup)
    print(f"[bench] timing {args.steps} steps", file=sys.stderr, flush=True)
    dt, nodes, tokens, depth = timed(sess, args.steps)
    value = nodes / dt
    prof = profile_pass(rt, abi, sess, args.profile_steps)
    # fixed max tree (depth 6, width 10, 60 nodes) for comparison
    fdt, fnodes = 1.0, 0
    if not args.no_fixed:
        sfix = fresh(fixed=True)
        run_steps(sfix, 3)
        fdt, fnodes, ftokens, _ = timed(sfix, min(args.steps, 50))
    g = prof["gemm"]
    gemm_avg_s = g["ms"] / max(g["launches"], 1) * 1e-3
    gemm_bytes = g["bytes"] / max(g["launches"], 1)
    gemm_gbs = gemm_bytes / gemm_avg_s / 1e9 if gemm_avg_s > 0 else 0.0
    a = prof["attn"]
    attn_gbs = a["bytes"] / (a["ms"] * 1e-3) / 1e9 if a["ms"] > 0 else 0.0
    micro = {} if args.no_microbench else attn_microbench(rt)
    compact = None if args.no_microbench else compact_microbench(rt)
    mfma = None if args.no_mfma else mfma_benchmark(rt)
    guided = None if args.no_guided else guided_run(min(args.steps, 50))
    stochastic = None if args.no_stochastic else stochastic_run(min(args.steps, 50))
    batched = None if args.no_batch else [batched_run(16, True, min(args.steps, 30)),
                                          batched_run(16, False, min(args.steps, 30))]
    line = {
        "metric": "verified draft-tree nodes/sec + tree-attn HBM GB/s (% peak), 1xMI355X",
        "value": round(value, 2),
        "unit": "nodes/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(dt / args.steps * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded random-init weights and prompt ids)",
        "config": {"workload": "LlamaGen-XL-shaped ADT-Tree cycle: 36 layers, d_model 1280, 20x64 heads, "
                               "FFN 3584, vocab 16384, 120-token prompt, 32x32 grid, trees <= 60 nodes, "
                               "width <= 10, depth <= 6, greedy, batch 1",
                   "tree": "ADT schedule (adjacent init + bisection)",
                   "mean_depth": round(depth / args.steps, 3), "tokens_per_step": round(tokens / args.steps, 3),
                   "nodes_per_step": round(nodes / args.steps, 2)},
        "roofline": {"bound": "hbm", "kernel": "gemm_tile_kernel (bf16 projections with fused epilogues)",
                     "achieved": round(gemm_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(gemm_gbs / HBM_PEAK_GBS, 4), "traffic": gemm_traffic(),
                     "launches": g["launches"], "avg_us": round(gemm_avg_s * 1e6, 3),
                     "bytes_per_launch": round(gemm_bytes)},
        "tree_attn": {"in_cycle_GB_s": round(attn_gbs, 1), "in_cycle_frac": round(attn_gbs / HBM_PEAK_GBS, 4),
                      "in_cycle_avg_us": round(a["ms"] / max(a["launches"], 1) * 1e3, 3),
                      "microbench_16x32x128": micro},
        "kv_compact": compact,
        "batched_verify_gemm": mfma,
        "guided": guided,
        "batched": batched,
        "stochastic_children": stochastic,
        "fixed_tree": {"nodes_per_s": round(fnodes / fdt, 2), "ms_per_step": round(fdt / min(args.steps, 50) * 1e3, 4),
                       "nodes_per_step": round(fnodes / min(args.steps, 50), 2), "tree": "depth 6, width 10, top-60"},
    }
    if not args.no_cpu:
        print("[bench] timing the CPU oracle", file=sys.stderr, flush=True)
        line["cpu_baseline"] = cpu_baseline(cfg, w, args.cpu_seconds)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
