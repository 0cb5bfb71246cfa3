"""The C ABI on the CPU: libadt.so loads, exports every entry point declared in
include/adt.h, validates arguments before launching anything, and its host-only schedule
matches the oracle's (Sec. 4.1-4.2, Eq. 2)."""
import ctypes as C
import json
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def L():
    from paper_2512_21857_amd import abi
    return abi.lib()


def declared_symbols():
    text = open(os.path.join(ROOT, "include", "adt.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(adt_[a-z0-9_]+)\s*\(", text)))


def test_exports_every_declared_symbol(L):
    from paper_2512_21857_amd import abi
    names = declared_symbols()
    assert len(names) >= 20
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(abi.EXPORTED)
    assert L.adt_version() == 1


def test_debug_build_exports_the_same_symbols(L):
    """libadt_debug.so (device invariant checks compiled in) has the same ABI; only it
    reports the checks as enabled."""
    from paper_2512_21857_amd import abi
    D = abi.lib_debug()
    for n in declared_symbols():
        assert hasattr(D, n), n
    assert D.adt_device_checks_enabled() == 1
    assert L.adt_device_checks_enabled() == 0
    assert abi.E_DEVICE_INVARIANT == -6 and abi.E_STATE == -7


def test_argument_errors_return_codes_without_launching(L):
    from paper_2512_21857_amd import abi
    assert L.adt_tree_attn(None, None, None, 0, 0, None, None, None, None, 1, 1, 64, 1, 1, 1.0, 1, None, None, 0,
                           None) == abi.E_ARG
    assert "null" in abi.last_error()
    fake = 0x1000
    # unsupported head size, oversize tree
    assert L.adt_tree_attn(fake, fake, fake, 0, 96 * 10, fake, fake, fake, fake, 1, 1, 96, 1, 10, 1.0, 1, fake, fake, 0,
                           None) == abi.E_SHAPE
    assert L.adt_tree_attn(fake, fake, fake, 0, 64 * 10, fake, fake, fake, fake, 1, 1, 64, 129, 10, 1.0, 1, fake, fake,
                           0, None) == abi.E_CAPACITY
    assert L.adt_kv_compact(fake, fake, 1, 1, 64, 0, 64, fake, fake, 4, fake, 200, 1, None) == abi.E_CAPACITY
    # 100 accepted fp32 rows of 1024 (400 KB per slice) exceed one block's staging
    assert L.adt_kv_compact(fake, fake, 1, 1, 1024, 0, 1024, fake, fake, 101, fake, 100, 0, None) == abi.E_UNSUPPORTED
    assert L.adt_tree_masks(fake, fake, 1, 300, fake, None, None) == abi.E_CAPACITY
    cfg = abi.AcceptCfg(7, 1.0, 0, 0.0, 1, 0, 0, None, 0)
    import ctypes as C
    assert L.adt_verify_accept(fake, 16, 16, fake, fake, fake, fake, 4, C.byref(cfg), 0, fake, fake, fake, fake, 1 << 20,
                               None) == abi.E_ARG
    # the exact and relaxed walks cover at most 65536 ids per row
    for mode in (abi.ACCEPT_EXACT, abi.ACCEPT_RELAXED):
        cfg = abi.AcceptCfg(mode, 1.0, 0, 0.1, 1, 0, 0, None, 0)
        assert L.adt_verify_accept(fake, 70000, 70000, fake, fake, fake, fake, 4, C.byref(cfg), 0, fake, fake, fake,
                                   fake, 1 << 30, None) == abi.E_UNSUPPORTED
    # stochastic-children acceptance without its q rows (null, short row stride, no rows)
    for q_logits, q_ld, q_row, q_rows in ((None, 16, fake, 4), (fake, 8, fake, 4), (fake, 16, None, 4),
                                          (fake, 16, fake, 0)):
        cfg = abi.AcceptCfg(abi.ACCEPT_MSS, 1.0, 0, 0.0, 1, 0, 0, None, 0, 2, q_logits, q_ld, q_row, q_rows)
        assert L.adt_verify_accept(fake, 16, 16, fake, fake, fake, fake, 4, C.byref(cfg), 0, fake, fake, fake, fake,
                                   1 << 20, None) == abi.E_ARG
    # batched projection: null operands; N not a multiple of 128, K not of 64, short leading dimension
    assert L.adt_gemm_bf16(None, 64, fake, 64, 8, 128, 64, fake, 128, None) == abi.E_ARG
    assert L.adt_gemm_bf16_packed(fake, 64, None, 8, 128, 64, fake, 128, None, 0, None) == abi.E_ARG
    assert L.adt_gemm_bf16_packed(fake, 64, fake, 8, 384, 96, fake, 384, None, 0, None) == abi.E_SHAPE
    assert L.adt_gemm_bf16_packed(fake, 64, fake, 0, 256, 64, fake, 256, None, 0, None) == abi.E_SHAPE
    # K split only for few blocks and long K: 4 ranges of the 64-block 4096 x 11008 product,
    # none for the 256-block LM head or shorter K
    assert L.adt_gemm_bf16_packed_workspace_size(976, 4096, 11008) == 3 * 976 * 4096 * 4
    assert L.adt_gemm_bf16_packed_workspace_size(976, 65536, 11008) == 0
    # 256 blocks of 128 x 128 fill the CUs: no split
    assert L.adt_gemm_bf16_packed_workspace_size(976, 4096, 4096) == 0
    # 80 blocks of 128 x 128 with K >= 2048: K split in two, one partial
    assert L.adt_gemm_bf16_packed_workspace_size(976, 1280, 3584) == 976 * 1280 * 4
    # 344 blocks of 256 x 256: the last 22 column blocks (88 blocks) split two ways
    assert L.adt_gemm_bf16_packed_workspace_size(976, 22016, 4096) == 976 * 22 * 256 * 4
    # 192 blocks of 256 x 256 become 256 of 384 x 128: no partials
    assert L.adt_gemm_bf16_packed_workspace_size(976, 12288, 4096) == 0
    assert L.adt_gemm_bf16_packed_workspace_size(976, 32000, 4096) == 0
    assert L.adt_gemm_bf16(fake, 64, fake, 64, 8, 100, 64, fake, 128, None) == abi.E_SHAPE
    assert L.adt_gemm_bf16(fake, 96, fake, 96, 8, 128, 96, fake, 128, None) == abi.E_SHAPE
    assert L.adt_gemm_bf16(fake, 32, fake, 64, 8, 128, 64, fake, 128, None) == abi.E_SHAPE
    sess = C.c_void_p()
    assert L.adt_session_create(None, None, C.byref(sess)) == abi.E_ARG
    assert L.adt_step(None, None, None) == abi.E_ARG


def test_schedule_matches_oracle(L):
    from paper_2512_21857_amd import runtime
    from synth import SchedCfg
    from oracle.schedule import schedule
    gold = json.load(open(os.path.join(ROOT, "tests", "golden", "schedule_trajectories.json")))
    for case in gold["cases"]:
        sc = SchedCfg(**case["sched"])
        s = runtime.sched_struct(sc)
        rec, prev = None, None
        for a, tree in zip(case["accepted"], case["trees"]):
            got = runtime.schedule_next(s, rec, prev, 10_000)
            assert list(got) == tree == list(schedule(sc, rec, prev, 10_000))
            rec, prev = got, (a, got[0])
    sc = SchedCfg(1, 6, 4, 10, 1, 10, 1.0, 60, 5, 10)
    s = runtime.sched_struct(sc)
    for left in [None, (1, 4), (6, 10), (3, 7)]:
        for prev in [None, (0, 3), (3, 3), (6, 6)]:
            for rem in (1, 2, 3, 50):
                if left is None and prev is not None:
                    continue
                assert runtime.schedule_next(s, left, prev, rem) == schedule(sc, left, prev, rem)


@pytest.mark.parametrize("rule", ["horizontal", "vertical", "random", "tokenflock", "fixed", "deep"])
def test_schedule_init_rules_match_oracle(L, rule):
    """adt_schedule_init + adt_schedule_next against the oracle's initial() + schedule() over
    random record tables (Sec. 4.1, Sec. 5.3 Eqs. 6-8, Table V, Sec. 4.2)."""
    import dataclasses
    from paper_2512_21857_amd import runtime
    from synth import SchedCfg
    from oracle.schedule import initial, schedule
    rng = np.random.default_rng(5)
    W, n = 7, 70
    base = SchedCfg(1, 6, 4, 10, 1, 10, 1.0, 60, 5, 10)
    kw = {"fixed": dict(fix_d=1, fix_k=25), "deep": dict(k_clamp="deep", init="vertical")}.get(rule, {"init": rule})
    for delta in ((1, 2, 3) if rule == "tokenflock" else (2,)):
        sc = dataclasses.replace(base, flock_delta=delta, seed=99, **kw)
        s = runtime.sched_struct(sc, W)
        for trial in range(40):
            cell = int(rng.integers(0, n))
            recs = {g: (int(rng.integers(0, 12)), int(rng.integers(0, 20)))
                    for g in range(1, n) if rng.random() < 0.8}
            init = runtime.schedule_init(s, cell, recs, n)
            assert init == initial(sc, cell, {g: r for g, r in recs.items() if g < cell}, W), (rule, cell)
            for prev in (None, (0, 2), (3, 3), (1, 1)):
                for rem in (1, 3, 50):
                    assert runtime.schedule_next(s, init, prev, rem) == schedule(sc, init, prev, rem)


def test_schedule_init_rejects_bad_settings(L):
    import dataclasses
    from paper_2512_21857_amd import runtime, abi
    from synth import SchedCfg
    base = SchedCfg(1, 6, 4, 10, 1, 10, 1.0, 60, 5, 10)
    rd = (C.c_int32 * 4)()
    out = [C.c_int32() for _ in range(3)]
    for kw, w in ((dict(init="vertical"), 0), (dict(init="tokenflock", flock_delta=0), 4),
                  (dict(k_clamp="deep", d_lo=2), 4), (dict(fix_d=-1), 4)):
        s = runtime.sched_struct(dataclasses.replace(base, **kw), w)
        assert L.adt_schedule_init(C.byref(s), 1, 4, rd, rd, rd, *[C.byref(o) for o in out]) == abi.E_ARG
    s = runtime.sched_struct(base, 4)
    s.init_mode = 7
    assert L.adt_schedule_init(C.byref(s), 1, 4, rd, rd, rd, *[C.byref(o) for o in out]) == abi.E_ARG
    s.init_mode = abi.INIT_HORIZONTAL
    assert L.adt_schedule_init(C.byref(s), 4, 4, rd, rd, rd, *[C.byref(o) for o in out]) == abi.E_ARG
    assert L.adt_schedule_init(C.byref(s), 0, 4, None, rd, rd, *[C.byref(o) for o in out]) == abi.E_ARG


def test_accept_cfg_keeps_its_tensors_alive():
    """The config struct holds raw device pointers; the binding keeps the tensors they point
    to alive with it, so temporaries passed in cannot be freed (and their memory reused)
    before a kernel reads them."""
    import gc
    import torch
    from paper_2512_21857_amd import runtime as rt
    cfg = rt.accept_cfg("mss", 1.0, 0, seed=1, children=2, q_logits=torch.arange(12.0).view(3, 4),
                        q_row=torch.tensor([0, 2], dtype=torch.int32))
    gc.collect()
    q_logits, q_row = cfg._tensors[1], cfg._tensors[2]
    assert cfg.q_logits == q_logits.data_ptr() and cfg.q_row == q_row.data_ptr()
    assert (cfg.q_ld, cfg.q_rows, cfg.children) == (4, 3, 2)
    assert q_logits[2, 3].item() == 11.0


def test_capture_arguments(L):
    """Layer-by-layer record: a null session is refused, a record without its metadata buffer
    is refused, and a null session has no records."""
    import ctypes as C
    from paper_2512_21857_amd import abi
    assert L.adt_session_set_capture(None, None) == abi.E_ARG
    assert L.adt_session_capture_count(None) == 0
    rec = abi.CaptureRec()
    assert L.adt_session_capture_record(None, 0, C.byref(rec)) == abi.E_ARG


def test_tree_attn_noalloc_rejects_oversize_partials(L):
    """Key-split partials beyond the library's 16 MiB scratch (120 pairs of 128-row trees at head
    size 128 over 10000 slots: 3 key ranges, 24 MB) are refused before anything is enqueued;
    argument errors are those of adt_tree_attn."""
    from paper_2512_21857_amd import abi
    fake = 0x1000
    assert L.adt_tree_attn_noalloc(fake, fake, fake, 0, 128 * 10000, fake, fake, fake, fake, 1, 120, 128, 128, 10000,
                                   1.0, abi.BF16, fake, None) == abi.E_CAPACITY
    assert "scratch" in abi.last_error()
    assert L.adt_tree_attn_noalloc(None, fake, fake, 0, 64, fake, fake, fake, fake, 1, 1, 64, 1, 1, 1.0, abi.BF16, fake,
                                   None) == abi.E_ARG
