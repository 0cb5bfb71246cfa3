#!/usr/bin/env python3
"""Throughput of the ADT-Tree draft-then-verify cycle on one MI355X.

A step is one adt_step call: ADT schedule, draft-tree expansion (draft forwards, top-k,
scoring, rerank), the tree-masked verification forward of the target model, acceptance, KV
compaction and commit.  The headline workload is the Lumina-mGPT-7B-shaped synthetic model
(32 layers, d_model 4096, 32 x 128 heads, SwiGLU 11008, vocab 65536, bf16, seeded
N(0, 0.02) weights), a 64-token seeded prompt and a 48 x 48 image grid with a row-end token
per row (2352 tokens, KV length up to ~2.4k), trees of at most 60 draft nodes with depth
1-8 and width 1-10 set per position by the ADT rule, its acceptance statistic drawn from a
seeded Poisson(lambda) table (lambda 4 / 1 on a checkerboard of 8 x 8 regions), greedy
acceptance, batch 1.  The K timed steps start at the middle of the image (KV length ~1240,
the image's mean), after W warm-up steps.

The metric is verified draft-tree nodes per second.  The line also carries: the roofline of
the dominant kernel (the weight-streaming projections); tree-attention bandwidth in the cycle
(mid-image and near the end, KV ~2.4k) and in the 16 x 32 x 128 microbenchmark; KV compaction
of random accepted paths; one whole image decoded; the Anole-7B-shaped workload with exact and
relaxed acceptance; the LlamaGen-XL-shaped and tiny workloads; the batched verify projections;
guided, stochastic-children and 16-image batched cycles; on-box bandwidth and MFMA probes; and
the CPU oracle timed on this host.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W]
"""
from __future__ import annotations

import argparse
import dataclasses
import hashlib
import json
import os
import subprocess
import sys
import time

import numpy as np

HBM_PEAK_GBS = 8000.0
MFMA_PEAK_TFLOPS = 2500.0
ROOT = os.path.dirname(os.path.abspath(__file__))
# the sources the GEMM kernel is compiled from (kernel, shared helpers, epilogue struct)
GEMM_SRCS = [os.path.join(ROOT, "paper_2512_21857_amd", "csrc", *parts)
             for parts in (("kernels", "gemm.hip"), ("common.h",), ("launch.h",))]
TRAFFIC_FILES = {"lumina_7b": os.path.join(ROOT, "profiles", "gemm_rows_lumina_7b_traffic.md")}


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def gemm_traffic(workload, algorithmic_bytes_per_launch):
    """HBM bytes per GEMM launch: the counter-measured traffic / algorithmic ratio of the
    committed FETCH_SIZE / WRITE_SIZE summary of this workload (every projection launch of a
    --traffic-run) times this run's algorithmic bytes per launch; None when the kernel's
    sources changed since the counters were taken (sha256 over gemm.hip, common.h and
    launch.h, in that order) or no summary exists."""
    try:
        text = open(TRAFFIC_FILES[workload]).read()
        h = hashlib.sha256()
        for path in GEMM_SRCS:
            h.update(open(path, "rb").read())
        src = h.hexdigest()
    except (OSError, KeyError):
        return None
    keys = ("source_sha256:", "traffic_over_algorithmic:")
    fields = dict(line.split(":", 1) for line in text.splitlines() if line.startswith(keys))
    if fields.get("source_sha256", "").strip() != src or "traffic_over_algorithmic" not in fields:
        return None
    return int(round(float(fields["traffic_over_algorithmic"].strip()) * algorithmic_bytes_per_launch))


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--profile-steps", type=int, default=30)
    ap.add_argument("--cpu-seconds", type=float, default=20.0)
    ap.add_argument("--headline-only", action="store_true", help="only the Lumina-7B-shaped lines")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--no-full-image", action="store_true")
    ap.add_argument("--no-anole", action="store_true")
    ap.add_argument("--no-small", action="store_true", help="skip the LlamaGen-XL and tiny workloads")
    ap.add_argument("--no-microbench", action="store_true")
    ap.add_argument("--no-mfma", action="store_true")
    ap.add_argument("--no-extras", action="store_true", help="skip guided / stochastic / batched cycles")
    ap.add_argument("--start-cell", type=int, default=-1, help="first timed image cell (default: mid-image)")
    ap.add_argument("--traffic-run", action="store_true",
                    help="counter-collection mode: profile every projection launch from the prefill on over the "
                         "warm-up and timed steps of the headline workload and print their count and algorithmic bytes")
    ap.add_argument("--microbench-run", action="store_true",
                    help="only the tree-attention and KV-compaction microbenchmarks (for counter collection)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="first copy 512 MiB device-to-device (a kernel of known traffic for counter scaling)")
    return ap.parse_args()


# ------------------------------------------------------------------------------ cycles
def run_steps(sess, k):
    import torch
    nodes = tokens = depth = steps = 0
    for _ in range(k):
        o = sess.step()
        if o["done"] and o["n_committed"] == 0:
            break
        nodes += o["n_nodes"] - 1
        tokens += o["n_committed"]
        depth += o["d_hat"]
        steps += 1
    torch.cuda.synchronize()
    return nodes, tokens, depth, steps


def timed(sess, k, tag=None):
    """k steps between two synchronisations; with a tag, the CLOCK_MONOTONIC window of the
    timed region goes to stderr for cutting a kernel trace of the same command."""
    import torch
    torch.cuda.synchronize()
    w0 = time.monotonic_ns()
    t0 = time.perf_counter()
    nodes, tokens, depth, steps = run_steps(sess, k)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    if tag:
        log(f"{tag} pass window {w0} {time.monotonic_ns()}")
    return dt, nodes, tokens, depth, steps


def fast_forward(sess, cfg, cell):
    """Untimed steps until the image cell of the next tree's first token reaches `cell`."""
    while True:
        v = sess.view()
        if v.L + 1 - cfg.prefix_len >= cell:
            return
        if sess.step()["done"]:
            return


def profile_pass(abi, sess, k, tag="profile"):
    """Per-kernel-class HIP-event timing over k further steps of the same session (eager).
    The pass's CLOCK_MONOTONIC window goes to stderr, so a kernel trace of the same command
    (whose timestamps use that clock) can be cut to the same launches."""
    import ctypes as C
    import torch
    L = abi.lib()
    abi.check(L.adt_profile_enable(1))
    for cls in (abi.PROF_GEMM, abi.PROF_ATTN, abi.PROF_COMPACT, abi.PROF_ROWS):
        L.adt_profile_read(cls, None, None, None, None, 1)
    v0 = sess.view()
    torch.cuda.synchronize()
    t0 = time.monotonic_ns()
    run_steps(sess, k)
    t1 = time.monotonic_ns()
    log(f"{tag} pass window {t0} {t1}")
    v1 = sess.view()
    out = {"L_from": v0.L, "L_to": v1.L}
    for name, cls in (("gemm", abi.PROF_GEMM), ("attn", abi.PROF_ATTN), ("compact", abi.PROF_COMPACT),
                      ("rows", abi.PROF_ROWS)):
        n, ms, by, fl = C.c_int64(), C.c_double(), C.c_double(), C.c_double()
        abi.check(L.adt_profile_read(cls, C.byref(n), C.byref(ms), C.byref(by), C.byref(fl), 1))
        out[name] = {"launches": n.value, "ms": ms.value, "bytes": by.value, "flops": fl.value}
    abi.check(L.adt_profile_enable(0))
    return out


def roofline_of(prof, workload, kernel):
    g = prof["gemm"]
    r = prof["rows"]
    avg_s = g["ms"] / max(g["launches"], 1) * 1e-3
    byts = g["bytes"] / max(g["launches"], 1)
    gbs = byts / avg_s / 1e9 if avg_s > 0 else 0.0
    return {"bound": "hbm", "kernel": kernel, "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": gemm_traffic(workload, byts), "launches": g["launches"],
            "avg_us": round(avg_s * 1e6, 3), "bytes_per_launch": round(byts),
            "residual_finish": {"launches": r["launches"], "avg_us": round(r["ms"] / max(r["launches"], 1) * 1e3, 3),
                                "kernel": "resid_norm_kernel (K-range sums + residual add + RMSNorm)"}}


def attn_of(prof):
    a = prof["attn"]
    gbs = a["bytes"] / (a["ms"] * 1e-3) / 1e9 if a["ms"] > 0 else 0.0
    return {"GB_s": round(gbs, 1), "frac": round(gbs / HBM_PEAK_GBS, 4), "launches": a["launches"],
            "avg_us": round(a["ms"] / max(a["launches"], 1) * 1e3, 3), "kv_len": [prof["L_from"], prof["L_to"]]}


def steps_line(dt, nodes, tokens, depth, steps):
    return {"nodes_per_s": round(nodes / dt, 2), "tokens_per_s": round(tokens / dt, 2),
            "ms_per_step": round(dt / max(steps, 1) * 1e3, 4), "nodes_per_step": round(nodes / max(steps, 1), 2),
            "tokens_per_step": round(tokens / max(steps, 1), 3), "mean_depth": round(depth / max(steps, 1), 3),
            "steps": steps}


def workload_run(rt, dm, cfg, pre, k, warm, start_cell, tag=None, **sess_kw):
    sess = rt.DeviceSession(dm, cfg, **sess_kw)
    sess.prefill(pre)
    fast_forward(sess, cfg, start_cell)
    run_steps(sess, warm)
    line = steps_line(*timed(sess, k, tag))
    line["start_cell"] = start_cell
    return sess, line


def full_image(rt, dm, cfg, pre, **sess_kw):
    """One whole image: prefill (untimed), then every cycle until the last grid cell."""
    import torch
    sess = rt.DeviceSession(dm, cfg, **sess_kw)
    sess.prefill(pre)
    run_steps(sess, 3)         # warm the graphs of the first tree shapes
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    nodes, tokens, depth, steps = run_steps(sess, 1 << 30)
    dt = time.perf_counter() - t0
    line = steps_line(dt, nodes, tokens, depth, steps)
    line["image_tokens"] = cfg.n_image
    return line


# ------------------------------------------------------------------------------ microbenchmarks
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
        out[str(n)] = {"us": round(ms * 1e3, 2), "GB_s": round(gbs, 1), "frac": round(gbs / HBM_PEAK_GBS, 4),
                       "bytes_per_launch": int(byts / iters)}
        del bufs, outs
        torch.cuda.empty_cache()
    return out


def compact_microbench(rt, B=16, heads=32, Dh=128, nodes=128, iters=50, seed=3):
    """KV compaction as the microbenchmark states it: 16 sequences of 32 heads x 128 (bf16),
    each moving a random accepted path of a ~ U{1..12} sorted distinct nodes of a 128-node
    tree (synth.compaction_paths).  Each call works at prefix lengths shifted so its rows are
    not in the last-level cache.  At <= 3.1 MB per call this is latency-bound."""
    import torch
    import synth
    rng = np.random.default_rng([seed, 40_000])
    base = rng.integers(512, 2401, size=B)
    step = nodes + 8
    S_cap = int(base.max()) + step * (iters + 3) + nodes
    gen = torch.Generator(device="cuda")
    gen.manual_seed(seed)
    k = torch.randn((B, heads, S_cap, Dh), generator=gen, device="cuda", dtype=torch.bfloat16)
    v = torch.randn((B, heads, S_cap, Dh), generator=gen, device="cuda", dtype=torch.bfloat16)
    calls = []
    for i in range(iters + 3):
        path, a = synth.compaction_paths(rng, np.full(B, nodes), a_max=12)
        calls.append((torch.from_numpy(path).cuda(), torch.from_numpy(a).cuda(),
                      torch.from_numpy((base + step * i).astype(np.int32)).cuda(), int(a.sum())))
    for i in range(3):
        c = calls[iters + i]
        rt.kv_compact(k, v, c[2], c[0], c[1], 12)
    st = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(st)
    rows = 0
    for i in range(iters):
        c = calls[i]
        rt.kv_compact(k, v, c[2], c[0], c[1], 12)
        rows += c[3]
    e1.record(st)
    e1.synchronize()
    ms = e0.elapsed_time(e1) / iters
    byts = 2.0 * 2 * heads * Dh * 2 * rows / iters     # K and V rows, each read once and written once
    gbs = byts / (ms * 1e-3) / 1e9
    del k, v
    torch.cuda.empty_cache()
    return {"us": round(ms * 1e3, 2), "GB_s": round(gbs, 1), "frac": round(gbs / HBM_PEAK_GBS, 4),
            "bytes": int(byts), "bound": "latency (a few MB per call)",
            "workload": f"{B} sequences x {heads} heads x {Dh} bf16, accepted path a ~ U{{1..12}} of a "
                        f"{nodes}-node tree per sequence (mean a = {rows / iters / B:.2f})"}


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


def onbox_probes(rt, read_bytes=4 << 30, iters=10):
    """What this device sustains: a streaming read of 4 GiB (the library's probe kernel) and a
    register-only MFMA loop, each timed with events, beside the nominal peaks."""
    import torch
    sink = rt.probe_sink()
    buf = torch.empty(read_bytes, dtype=torch.uint8, device="cuda")
    buf.fill_(1)
    st = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    for _ in range(2):
        rt.probe_hbm_read(buf, sink)
    e0.record(st)
    for _ in range(iters):
        rt.probe_hbm_read(buf, sink)
    e1.record(st)
    e1.synchronize()
    rd = read_bytes * iters / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del buf
    rt.probe_mfma(200, sink)
    e0.record(st)
    fl = 0.0
    for _ in range(iters):
        fl += rt.probe_mfma(2000, sink)
    e1.record(st)
    e1.synchronize()
    tf = fl / (e0.elapsed_time(e1) * 1e-3) / 1e12
    torch.cuda.empty_cache()
    return {"hbm_read_GB_s": round(rd, 1), "hbm_nominal_GB_s": HBM_PEAK_GBS,
            "hbm_read_frac_of_nominal": round(rd / HBM_PEAK_GBS, 4),
            "mfma_bf16_TFLOP_s": round(tf, 1), "mfma_bf16_nominal_TFLOP_s": MFMA_PEAK_TFLOPS,
            "mfma_frac_of_nominal": round(tf / MFMA_PEAK_TFLOPS, 4),
            "probes": "adt_probe_hbm_read (16-byte nontemporal loads over 4 GiB), adt_probe_mfma "
                      "(back-to-back 32x32x16 bf16 MFMAs, register operands)"}


# ------------------------------------------------------------------------------ CPU oracle
def cpu_model():
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for line in out.splitlines():
            if line.startswith("Model name:"):
                return line.split(":", 1)[1].strip()
    except Exception:
        pass
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(cfg, weights, budget_s, poisson=None):
    """The oracle as it stands, on this host's cores, over the first cycles of the same
    workload: prefill untimed, then cycles until the budget is spent (at least one)."""
    from threadpoolctl import threadpool_info, threadpool_limits
    from oracle.decode import Decoder
    from oracle.model import OracleModel
    import synth
    cores = len(os.sched_getaffinity(0))
    with threadpool_limits(limits=cores):
        om = OracleModel(cfg, weights)
        dec = Decoder(cfg, om, synth.prefix_ids(cfg), poisson=poisson)
        t0 = time.perf_counter()
        dec.prefill()
        t_pre = time.perf_counter() - t0
        nodes = steps = 0
        t0 = time.perf_counter()
        while (steps == 0 or time.perf_counter() - t0 < budget_s) and not dec.done():
            info = dec.step()
            nodes += info.tree.n - 1
            steps += 1
        dt = time.perf_counter() - t0
        blas = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    return {"value": round(nodes / dt, 3), "unit": "nodes/s", "cores": int(cores), "blas_threads": int(blas),
            "cpu_model": cpu_model(), "kind": "oracle", "s_per_step": round(dt / steps, 3),
            "sample": f"fp64 NumPy oracle on {cfg.name}: prefill ({t_pre:.1f} s, untimed) then the first {steps} "
                      f"ADT cycles ({nodes} draft nodes) in {dt:.1f} s"}


# ------------------------------------------------------------------------------ main
def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "the library runs on one GPU only; use --gpus 1"}))
        sys.exit(2)
    import torch
    sys.path.insert(0, ROOT)
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
    threads = min(16, len(os.sched_getaffinity(0)))
    K, W = args.steps, args.warmup
    if args.microbench_run:
        log("microbenchmarks only")
        print(json.dumps({"microbench_run": True, "tree_attn_16x32x128": attn_microbench(rt),
                          "kv_compact": compact_microbench(rt)}), flush=True)
        return

    # ---- headline: Lumina-mGPT-7B-shaped, Poisson-driven ADT trees, greedy, batch 1
    cfg = synth.get_config("lumina_7b")
    log(f"generating weights for {cfg.name}")
    w = synth.model_weights(cfg, threads=threads)
    dm = rt.DeviceModel(cfg, w)
    pre = synth.prefix_ids(cfg)
    poisson = synth.poisson_table(cfg)
    mid = cfg.n_image // 2 if args.start_cell < 0 else args.start_cell
    if args.traffic_run:
        import ctypes as C
        L = abi.lib()
        abi.check(L.adt_profile_enable(1))
        L.adt_profile_read(abi.PROF_GEMM, None, None, None, None, 1)
        L.adt_profile_read(abi.PROF_ATTN, None, None, None, None, 1)
        sess = rt.DeviceSession(dm, cfg, poisson=poisson)
        sess.prefill(pre)
        fast_forward(sess, cfg, mid)
        run_steps(sess, W + K)
        n, ms, by, fl = C.c_int64(), C.c_double(), C.c_double(), C.c_double()
        abi.check(L.adt_profile_read(abi.PROF_GEMM, C.byref(n), C.byref(ms), C.byref(by), C.byref(fl), 1))
        na, ba = C.c_int64(), C.c_double()
        abi.check(L.adt_profile_read(abi.PROF_ATTN, C.byref(na), C.byref(ms), C.byref(ba), C.byref(fl), 1))
        abi.check(L.adt_profile_enable(0))
        print(json.dumps({"traffic_run": cfg.name, "gemm_launches": n.value, "gemm_algorithmic_bytes": by.value,
                          "attn_calls": na.value, "attn_algorithmic_bytes": ba.value,
                          "start_cell": mid, "steps": W + K}), flush=True)
        return
    log(f"{cfg.name}: fast-forward to cell {mid}, {W} warm-up steps, {K} timed steps")
    sess, head = workload_run(rt, dm, cfg, pre, K, W, mid, tag="timed", poisson=poisson)
    prof_mid = profile_pass(abi, sess, args.profile_steps, "mid-image profile")
    fast_forward(sess, cfg, cfg.n_image - 2 * args.profile_steps)
    prof_end = profile_pass(abi, sess, args.profile_steps, "end-of-image profile")
    del sess
    full = None if args.no_full_image else full_image(rt, dm, cfg, pre, poisson=poisson)
    cpu = None
    if not args.no_cpu:
        log("timing the CPU oracle on the headline workload")
        cpu = cpu_baseline(cfg, w, args.cpu_seconds, poisson=poisson)
    del dm, w
    torch.cuda.empty_cache()

    line = {
        "metric": "verified draft-tree nodes/sec + tree-attn HBM GB/s (% peak), 1xMI355X",
        "value": head["nodes_per_s"],
        "unit": "nodes/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded random-init weights, prompt ids and Poisson acceptance table)",
        "config": {"workload": "Lumina-mGPT-7B-shaped ADT-Tree cycle: 32 layers, d_model 4096, 32x128 heads, "
                               "FFN 11008, vocab 65536, 64-token prompt, 48x48 grid + row-end column (2352 "
                               "tokens), trees <= 60 draft nodes, depth 1-8, width 1-10 set by the ADT rule "
                               "driven by a Poisson(lambda in {1,4}) checkerboard of 8x8 regions, greedy, batch 1",
                   "timed_from_cell": mid, "tokens_per_step": head["tokens_per_step"],
                   "nodes_per_step": head["nodes_per_step"], "mean_depth": head["mean_depth"],
                   "tokens_per_s": head["tokens_per_s"]},
        "roofline": roofline_of(prof_mid, "lumina_7b", "gemm_rows_kernel (bf16 projections, fused epilogues or K-range sums)"),
        "tree_attn": {"in_cycle_mid_image": attn_of(prof_mid), "in_cycle_end_of_image": attn_of(prof_end)},
        "full_image": full,
    }
    if cpu is not None:
        line["cpu_baseline"] = cpu

    if not args.headline_only:
        line["on_box_peaks"] = onbox_probes(rt)
        if not args.no_anole:
            acfg = synth.get_config("anole_7b", mode="exact")
            log(f"generating weights for {acfg.name}")
            aw = synth.model_weights(acfg, threads=threads)
            adm = rt.DeviceModel(acfg, aw)
            del aw
            apre = synth.prefix_ids(acfg)
            knn = rt.codebook_knn(torch.from_numpy(synth.codebook(acfg)).cuda(), 100)
            res = {}
            for mode in ("exact", "relaxed"):
                mcfg = synth.get_config("anole_7b", mode=mode)
                s, r = workload_run(rt, adm, mcfg, apre, min(K, 100), W, mcfg.n_image // 2,
                                    tag=f"anole {mode} timed", knn=knn if mode == "relaxed" else None)
                del s
                res[mode] = r
            line["anole_7b"] = {"workload": "Anole-7B-shaped: 32 layers, d 4096, 32x128 heads, FFN 11008, vocab "
                                            "65536 with 8192 image codes, 32x32 grid, T = 1, top-k 2000, trees "
                                            "<= 60 nodes; relaxed: k = 100 cosine codebook neighbours, delta 0.1",
                                **res}
            del adm, knn
            torch.cuda.empty_cache()
        if not args.no_small:
            lcfg = synth.get_config("llamagen_xl")
            log(f"generating weights for {lcfg.name}")
            lw = synth.model_weights(lcfg, threads=threads)
            ldm = rt.DeviceModel(lcfg, lw)
            lpre = synth.prefix_ids(lcfg)
            s, r = workload_run(rt, ldm, lcfg, lpre, min(K, 100), W, lcfg.n_image // 2, tag="llamagen timed")
            lprof = profile_pass(abi, s, args.profile_steps, "llamagen profile")
            del s
            s, fr = workload_run(rt, ldm, lcfg, lpre, min(K, 50), 3, lcfg.n_image // 2, fixed_tree=True)
            del s
            r["roofline"] = roofline_of(lprof, "llamagen_xl", "gemm_rows_kernel")
            r["tree_attn_in_cycle"] = attn_of(lprof)
            r["fixed_tree_depth6_width10"] = fr
            line["llamagen_xl"] = r
            if not args.no_extras:
                line["llamagen_xl"]["guided"] = guided_run(rt, ldm, lcfg, lpre, min(K, 50))
                line["llamagen_xl"]["stochastic_children"] = stochastic_run(rt, ldm, lcfg, lpre, min(K, 50))
                line["llamagen_xl"]["batched"] = [batched_run(rt, ldm, lcfg, 16, True, min(K, 30)),
                                                  batched_run(rt, ldm, lcfg, 16, False, min(K, 30))]
            del ldm, lw
            torch.cuda.empty_cache()
            tcfg = synth.get_config("tiny")
            tdm = rt.DeviceModel(tcfg, synth.model_weights(tcfg))
            line["tiny"] = full_image(rt, tdm, tcfg, synth.prefix_ids(tcfg))
            del tdm
        if not args.no_microbench:
            log("microbenchmarks")
            line["tree_attn"]["microbench_16x32x128"] = attn_microbench(rt)
            line["kv_compact"] = compact_microbench(rt)
        if not args.no_mfma:
            line["batched_verify_gemm"] = mfma_benchmark(rt)
    print(json.dumps(line), flush=True)


def guided_run(rt, dm, cfg, pre, k):
    """The cycle with classifier-free guidance (scale 3.0, conditional and unconditional
    branches in every forward)."""
    import synth
    gcfg = dataclasses.replace(cfg, guidance=3.0)
    gs = rt.DeviceSession(dm, gcfg)
    gs.prefill(pre, synth.null_prefix_ids(gcfg))
    run_steps(gs, 3)
    r = steps_line(*timed(gs, k))
    r["scale"] = 3.0
    return r


def stochastic_run(rt, dm, cfg, pre, k, children=3):
    """The cycle with stochastic children (drawn from q at T = 1, every drawn child kept,
    Eq. 1 acceptance with the residual norm(max(0, p - q)))."""
    import synth
    scfg = dataclasses.replace(cfg, accept=synth.AcceptCfg(mode="mss", temperature=1.0, top_k=0, children=children))
    ss = rt.DeviceSession(dm, scfg)
    ss.prefill(pre)
    run_steps(ss, 3)
    r = steps_line(*timed(ss, k))
    r["children"] = children
    return r


def batched_run(rt, dm, cfg, B, fixed, k):
    """B images decoded together: per image its own schedule and draft tree, one verify
    forward over the packed rows of all B trees per step (packed-weight MFMA GEMMs)."""
    import torch
    import synth
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
            "rows_per_step": round((nodes + B * k) / k, 1), "tokens_per_step": round(tokens / k, 3), "steps": k}


if __name__ == "__main__":
    main()
