"""ctypes declarations of the C ABI in include/adt.h (argument marshalling only).

The shared library is loaded after torch so that it binds to the HIP runtime torch has
already loaded (one runtime per process).  There is no fallback: if libadt.so is missing
every call raises."""
from __future__ import annotations

import ctypes as C
import os
from typing import Optional

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libadt.so")
DEBUG_LIB_PATH = os.path.join(PKG, "libadt_debug.so")   # device invariant checks compiled in

OK = 0
E_ARG, E_SHAPE, E_CAPACITY, E_HIP, E_UNSUPPORTED, E_DEVICE_INVARIANT, E_STATE = -1, -2, -3, -4, -5, -6, -7
F32, BF16 = 0, 1
MAX_NODES = 128
MASK_WORDS = 2
ACCEPT_GREEDY, ACCEPT_EXACT, ACCEPT_RELAXED, ACCEPT_MSS = 0, 1, 2, 3
PACK_STACK, PACK_GATE_UP, PACK_QKV = 0, 1, 2
ALPHA_REAL, ALPHA_POISSON = 0, 1
INIT_HORIZONTAL, INIT_VERTICAL, INIT_RANDOM, INIT_TOKENFLOCK = 0, 1, 2, 3
KCLAMP_ALWAYS, KCLAMP_DEEP = 0, 1
MAX_WIDTH = 16

p = C.c_void_p
i32 = C.c_int32
i64 = C.c_int64
u64 = C.c_uint64
f32 = C.c_float
sz = C.c_size_t
ip = C.POINTER(C.c_int32)


class AcceptCfg(C.Structure):
    _fields_ = [("mode", i32), ("temperature", f32), ("top_k", i32), ("delta", f32), ("knn_k", i32),
                ("knn_rows", i32), ("knn_stride", i32), ("knn", p), ("seed", u64), ("children", i32),
                ("q_logits", p), ("q_ld", i64), ("q_row", p), ("q_rows", i32)]


class SchedCfg(C.Structure):
    _fields_ = [("d_lo", i32), ("d_hi", i32), ("k_lo", i32), ("k_hi", i32), ("l_d", i32), ("l_k", i32),
                ("beta", f32), ("n_budget", i32), ("d0", i32), ("k0", i32), ("alpha_source", i32),
                ("init_mode", i32), ("grid_w", i32), ("flock_delta", i32), ("fix_d", i32), ("fix_k", i32),
                ("k_clamp", i32), ("seed", u64)]


class ModelDesc(C.Structure):
    _fields_ = [("n_layers", i32), ("d_model", i32), ("n_heads", i32), ("head_dim", i32), ("ffn", i32),
                ("vocab", i32), ("dtype", i32), ("rope_theta", f32), ("norm_eps", f32), ("embed", p),
                ("lm_head", p), ("draft_fc", p), ("w_qkv", C.POINTER(p)), ("w_o", C.POINTER(p)),
                ("w_gu", C.POINTER(p)), ("w_down", C.POINTER(p))]


class SessionDesc(C.Structure):
    _fields_ = [("prefix_len", i32), ("n_image", i32), ("s_cap", i32), ("k_cache", p), ("v_cache", p),
                ("dk_cache", p), ("dv_cache", p), ("allowed", ip), ("sched", SchedCfg), ("accept", AcceptCfg),
                ("poisson", ip), ("fixed_tree", i32), ("draft_table", p), ("draft_table_rows", i32),
                ("use_graphs", i32), ("guided", i32), ("guidance_scale", f32), ("workspace", p),
                ("workspace_bytes", sz)]


class StepOut(C.Structure):
    _fields_ = [("step", i32), ("d_hat", i32), ("k_hat", i32), ("n_nodes", i32), ("n_accepted", i32),
                ("n_committed", i32), ("tokens", i32 * MAX_NODES), ("done", i32)]


class SessionView(C.Structure):
    _fields_ = [("L", i32), ("Ld", i32), ("step", i32), ("n_tokens", i32), ("n_nodes", i32),
                ("logits", p), ("feat", p), ("draft_logits", p), ("parent", p), ("token", p), ("depth", p),
                ("score", p), ("mask", p), ("allowed_rows", p), ("path", p), ("n_acc", p), ("bonus", p),
                ("tokens_host", ip), ("q", p), ("att", p), ("act", p), ("resid", p), ("n_branches", i32),
                ("branch_logits", p), ("draft_branch_logits", p), ("logits_lo", i32), ("logits_hi", i32)]


class Capture(C.Structure):
    _fields_ = [("resid", p), ("resid_elems", sz), ("xin", p), ("xin_bytes", sz), ("meta", p), ("meta_elems", sz)]


class CaptureRec(C.Structure):
    _fields_ = [("draft", i32), ("nodes", i32), ("rows", i32), ("kv_prefix", i32), ("slot0", i32), ("n_tail", i32),
                ("snapshots", i32), ("resid_off", i64), ("xin_off", i64), ("meta_off", i64)]


_SIGS = {
    "adt_version": (i32, []),
    "adt_device_checks_enabled": (i32, []),
    "adt_device_check": (i32, [p]),
    "adt_last_error": (sz, [C.c_char_p, sz]),
    "adt_tree_attn_workspace_size": (sz, [i32, i32, i32, i32, i32]),
    "adt_tree_attn": (i32, [p, p, p, i64, i64, p, p, p, p, i32, i32, i32, i32, i32, f32, i32, p, p, sz, p]),
    "adt_tree_attn_noalloc": (i32, [p, p, p, i64, i64, p, p, p, p, i32, i32, i32, i32, i32, f32, i32, p, p]),
    "adt_tree_masks": (i32, [p, p, i32, i32, p, p, p]),
    "adt_kv_compact": (i32, [p, p, i32, i32, i32, i64, i64, p, p, i32, p, i32, i32, p]),
    "adt_accept_workspace_size": (sz, [i32]),
    "adt_verify_accept": (i32, [p, i64, i32, p, p, p, p, i32, C.POINTER(AcceptCfg), u64, p, p, p, p, sz, p]),
    "adt_codebook_knn_workspace_size": (sz, [i32]),
    "adt_codebook_knn": (i32, [p, i32, i32, i32, p, p, sz, p]),
    "adt_gemm_bf16": (i32, [p, i64, p, i64, i32, i32, i32, p, i64, p]),
    "adt_gemm_bf16_packed": (i32, [p, i64, p, i32, i32, i32, p, i64, p, sz, p]),
    "adt_gemm_bf16_packed_workspace_size": (sz, [i32, i32, i32]),
    "adt_packed_bytes": (sz, [i32, i32, i32]),
    "adt_pack_weight": (i32, [C.POINTER(p), ip, i32, i32, i32, i32, i32, p, p]),
    "adt_schedule_next": (i32, [C.POINTER(SchedCfg), i32, i32, i32, i32, i32, i32, i32, ip, ip]),
    "adt_schedule_init": (i32, [C.POINTER(SchedCfg), i32, i32, ip, ip, ip, ip, ip, ip]),
    "adt_model_create": (i32, [C.POINTER(ModelDesc), C.POINTER(p)]),
    "adt_model_destroy": (None, [p]),
    "adt_session_workspace_size": (sz, [p, C.POINTER(SessionDesc)]),
    "adt_session_create": (i32, [p, C.POINTER(SessionDesc), C.POINTER(p)]),
    "adt_session_destroy": (None, [p]),
    "adt_session_prefill": (i32, [p, ip, ip, p]),
    "adt_session_get_view": (i32, [p, C.POINTER(SessionView)]),
    "adt_session_set_capture": (i32, [p, C.POINTER(Capture)]),
    "adt_session_capture_count": (i32, [p]),
    "adt_session_capture_record": (i32, [p, i32, C.POINTER(CaptureRec)]),
    "adt_tree_expand": (i32, [p, i32, i32, i32, ip, p]),
    "adt_session_set_tree": (i32, [p, ip, ip, i32, p]),
    "adt_verify_forward": (i32, [p, p]),
    "adt_session_accept_commit": (i32, [p, i32, i32, C.POINTER(StepOut), p]),
    "adt_step": (i32, [p, C.POINTER(StepOut), p]),
    "adt_batch_workspace_size": (sz, [C.POINTER(p), i32]),
    "adt_batch_create": (i32, [C.POINTER(p), i32, p, sz, C.POINTER(p)]),
    "adt_batch_destroy": (None, [p]),
    "adt_batch_step": (i32, [p, C.POINTER(StepOut), p]),
    "adt_profile_enable": (i32, [i32]),
    "adt_probe_sink_bytes": (sz, []),
    "adt_probe_hbm_read": (i32, [p, sz, p, sz, p]),
    "adt_probe_mfma": (i32, [i32, p, sz, C.POINTER(C.c_double), p]),
    "adt_probe_sample_weights": (i32, [p, C.c_int64, p, p]),
    "adt_profile_read": (i32, [i32, C.POINTER(i64), C.POINTER(C.c_double), C.POINTER(C.c_double),
                               C.POINTER(C.c_double), i32]),
}

PROF_GEMM, PROF_ATTN, PROF_COMPACT, PROF_ROWS = 0, 1, 2, 3

EXPORTED = tuple(_SIGS)

_lib: Optional[C.CDLL] = None
_lib_debug: Optional[C.CDLL] = None


class AdtError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"ADT error {code}: {msg}")
        self.code = code


def _load(path: str) -> C.CDLL:
    import torch  # noqa: F401  (binds the library to the HIP runtime torch loaded)
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built; run paper_2512_21857_amd.build.build()")
    L = C.CDLL(path)
    for name, (res, args) in _SIGS.items():
        fn = getattr(L, name)
        fn.restype = res
        fn.argtypes = args
    return L


def lib() -> C.CDLL:
    global _lib
    if _lib is None:
        _lib = _load(LIB_PATH)
    return _lib


def lib_debug() -> C.CDLL:
    """The debug build (device invariant checks); its own error message buffer is read with
    last_error(lib_debug())."""
    global _lib_debug
    if _lib_debug is None:
        _lib_debug = _load(DEBUG_LIB_PATH)
    return _lib_debug


def last_error(L: Optional[C.CDLL] = None) -> str:
    buf = C.create_string_buffer(512)
    (L or lib()).adt_last_error(buf, 512)
    return buf.value.decode(errors="replace")


def check(code: int) -> None:
    if code != OK:
        raise AdtError(code, last_error())
