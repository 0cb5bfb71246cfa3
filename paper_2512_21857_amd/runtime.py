"""Python side of the C ABI: torch owns device memory (weights, caches, workspaces) and the
current HIP stream; every step of the hot path runs inside libadt.so.  These wrappers only
marshal pointers, sizes and structs."""
from __future__ import annotations

import ctypes as C
from typing import Dict, List, Optional, Sequence

import numpy as np
import torch

from . import abi
from .abi import check, lib

DTYPES = {"f32": abi.F32, "bf16": abi.BF16}
TORCH_DT = {abi.F32: torch.float32, abi.BF16: torch.bfloat16}


def _stream() -> C.c_void_p:
    return C.c_void_p(torch.cuda.current_stream().cuda_stream)


def _p(t: Optional[torch.Tensor]):
    return None if t is None else C.c_void_p(t.data_ptr())


def _require_cuda(*ts: torch.Tensor) -> None:
    for t in ts:
        if t is not None and not t.is_cuda:
            raise ValueError("device tensors expected")


def upload(arr: np.ndarray, device="cuda") -> torch.Tensor:
    """uint16 arrays are bfloat16 bit patterns; float32 stays float32."""
    if arr.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).to(device).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float32)).to(device)


# ============================================================================ standalone calls
def tree_attn(q: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor, kv_len: torch.Tensor,
              n_q: torch.Tensor, n_tail: torch.Tensor, mask: torch.Tensor, kv_cap: int,
              scale: Optional[float] = None, out: Optional[torch.Tensor] = None,
              workspace: Optional[torch.Tensor] = None) -> torch.Tensor:
    """q [B][nq_max][H][Dh]; caches [B][H][S_cap][Dh]; kv_len/n_q/n_tail int32 [B];
    mask uint64-as-int64 [B][nq_max][2]."""
    _require_cuda(q, k_cache, v_cache, kv_len, n_q, n_tail, mask)
    B, nq_max, H, Dh = q.shape
    S_cap = k_cache.shape[2]
    dt = abi.BF16 if q.dtype == torch.bfloat16 else abi.F32
    out = torch.empty_like(q) if out is None else out
    ws_bytes = lib().adt_tree_attn_workspace_size(B, H, Dh, nq_max, kv_cap)
    if workspace is None:
        workspace = torch.empty(max(ws_bytes, 256), dtype=torch.uint8, device=q.device)
    scale = 1.0 / float(np.sqrt(Dh)) if scale is None else scale
    check(lib().adt_tree_attn(_p(q), _p(k_cache), _p(v_cache), H * S_cap * Dh, S_cap * Dh, _p(kv_len), _p(n_q),
                              _p(n_tail), _p(mask), B, H, Dh, nq_max, kv_cap, scale, dt, _p(out), _p(workspace),
                              workspace.numel(), _stream()))
    return out


def tree_attn_noalloc(q: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor, kv_len: torch.Tensor,
                      n_q: torch.Tensor, n_tail: torch.Tensor, mask: torch.Tensor, kv_cap: int,
                      scale: Optional[float] = None, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """tree_attn through adt_tree_attn_noalloc (the library's own scratch, no workspace)."""
    _require_cuda(q, k_cache, v_cache, kv_len, n_q, n_tail, mask)
    B, nq_max, H, Dh = q.shape
    S_cap = k_cache.shape[2]
    dt = abi.BF16 if q.dtype == torch.bfloat16 else abi.F32
    out = torch.empty_like(q) if out is None else out
    scale = 1.0 / float(np.sqrt(Dh)) if scale is None else scale
    check(lib().adt_tree_attn_noalloc(_p(q), _p(k_cache), _p(v_cache), H * S_cap * Dh, S_cap * Dh, _p(kv_len), _p(n_q),
                                      _p(n_tail), _p(mask), B, H, Dh, nq_max, kv_cap, scale, dt, _p(out), _stream()))
    return out


def probe_hbm_read(buf: torch.Tensor, sink: torch.Tensor) -> None:
    """One streaming read of buf (device, 16-byte multiple) by the library's probe kernel."""
    _require_cuda(buf, sink)
    check(lib().adt_probe_hbm_read(_p(buf), buf.numel() * buf.element_size(), _p(sink), sink.numel(), _stream()))


def probe_mfma(iters: int, sink: torch.Tensor) -> float:
    """Launches the MFMA-only probe; returns the flops it performs."""
    _require_cuda(sink)
    fl = C.c_double()
    check(lib().adt_probe_mfma(iters, _p(sink), sink.numel(), C.byref(fl), _stream()))
    return fl.value


def probe_sink() -> torch.Tensor:
    return torch.empty(lib().adt_probe_sink_bytes(), dtype=torch.uint8, device="cuda")


def tree_masks(parent: torch.Tensor, n_nodes: torch.Tensor, depth: bool = True):
    """parent int32 [B][n_max] -> (mask int64 [B][n_max][2] holding uint64 bits, depth int32 [B][n_max])."""
    _require_cuda(parent, n_nodes)
    B, n_max = parent.shape
    mask = torch.empty(B, n_max, 2, dtype=torch.int64, device=parent.device)
    dep = torch.empty(B, n_max, dtype=torch.int32, device=parent.device) if depth else None
    check(lib().adt_tree_masks(_p(parent), _p(n_nodes), B, n_max, _p(mask), _p(dep), _stream()))
    return mask, dep


def kv_compact(k_cache: torch.Tensor, v_cache: torch.Tensor, kv_len: torch.Tensor, path: torch.Tensor,
               n_acc: torch.Tensor, a_max: int) -> None:
    """In place on caches [B][slices][S_cap][Dh]; path int32 [B][stride] (path[b][0] = 0)."""
    _require_cuda(k_cache, v_cache, kv_len, path, n_acc)
    B, slices, S_cap, Dh = k_cache.shape
    dt = abi.BF16 if k_cache.dtype == torch.bfloat16 else abi.F32
    check(lib().adt_kv_compact(_p(k_cache), _p(v_cache), B, slices, Dh, slices * S_cap * Dh, S_cap * Dh, _p(kv_len),
                               _p(path), path.shape[1], _p(n_acc), a_max, dt, _stream()))


def accept_cfg(mode: str = "greedy", temperature: float = 1.0, top_k: int = 0, delta: float = 0.0,
               knn: Optional[torch.Tensor] = None, knn_k: int = 1, seed: int = 0, children: int = 0,
               q_logits: Optional[torch.Tensor] = None, q_row: Optional[torch.Tensor] = None) -> abi.AcceptCfg:
    """mode 'mss': Eq. 1 with stochastic children (children per expanded node in a session;
    for adt_verify_accept the draft logit rows q_logits [rows][V] and the row q_row[u] that
    drew node u's children)."""
    m = {"greedy": abi.ACCEPT_GREEDY, "exact": abi.ACCEPT_EXACT, "relaxed": abi.ACCEPT_RELAXED,
         "mss": abi.ACCEPT_MSS}[mode]
    rows, stride = (knn.shape[0], knn.shape[1]) if knn is not None else (0, 0)
    q_ld, q_rows = (q_logits.stride(0), q_logits.shape[0]) if q_logits is not None else (0, 0)
    cfg = abi.AcceptCfg(m, temperature, top_k, delta, knn_k, rows, stride, _p(knn), seed, children, _p(q_logits),
                        q_ld, _p(q_row), q_rows)
    # the struct holds raw device pointers: keep their tensors alive as long as the struct
    cfg._tensors = (knn, q_logits, q_row)
    return cfg


def verify_accept(logits: torch.Tensor, parent: torch.Tensor, token: torch.Tensor, allowed: torch.Tensor,
                  n_nodes: torch.Tensor, cfg: abi.AcceptCfg, step: int, workspace: Optional[torch.Tensor] = None):
    """logits fp32 [n_max][V].  Returns device tensors (path [MAX_NODES], n_acc [1], bonus [1])."""
    _require_cuda(logits, parent, token, allowed, n_nodes)
    n_max, V = logits.shape
    dev = logits.device
    path = torch.zeros(abi.MAX_NODES, dtype=torch.int32, device=dev)
    n_acc = torch.zeros(1, dtype=torch.int32, device=dev)
    bonus = torch.zeros(1, dtype=torch.int32, device=dev)
    if workspace is None:
        workspace = torch.empty(lib().adt_accept_workspace_size(V), dtype=torch.uint8, device=dev)
    check(lib().adt_verify_accept(_p(logits), logits.stride(0), V, _p(parent), _p(token), _p(allowed), _p(n_nodes),
                                  n_max, C.byref(cfg), step, _p(path), _p(n_acc), _p(bonus), _p(workspace),
                                  workspace.numel(), _stream()))
    return path, n_acc, bonus


def gemm_bf16(x: torch.Tensor, w: torch.Tensor, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """x bf16 [M][K], w bf16 [N][K] (rows K-contiguous) -> fp32 [M][N] = x . w^T."""
    _require_cuda(x, w)
    assert x.dtype == torch.bfloat16 and w.dtype == torch.bfloat16 and x.stride(1) == 1 and w.stride(1) == 1
    M, K = x.shape
    N = w.shape[0]
    out = torch.empty(M, N, dtype=torch.float32, device=x.device) if out is None else out
    check(lib().adt_gemm_bf16(_p(x), x.stride(0), _p(w), w.stride(0), M, N, K, _p(out), out.stride(0), _stream()))
    return out


def pack_bf16(w: torch.Tensor) -> torch.Tensor:
    """w bf16 [N][K] (row-major, K contiguous) -> the library's packed tile layout (uint8 bytes)."""
    _require_cuda(w)
    assert w.dtype == torch.bfloat16 and w.is_contiguous()
    N, K = w.shape
    out = torch.empty(lib().adt_packed_bytes(N, K, abi.BF16), dtype=torch.uint8, device=w.device)
    srcs = (C.c_void_p * 1)(w.data_ptr())
    rows = (C.c_int32 * 1)(N)
    check(lib().adt_pack_weight(srcs, rows, 1, K, abi.PACK_STACK, 0, abi.BF16, _p(out), _stream()))
    return out


def gemm_bf16_packed(x: torch.Tensor, wp: torch.Tensor, N: int, out: Optional[torch.Tensor] = None,
                     workspace: Optional[torch.Tensor] = None, split: bool = True) -> torch.Tensor:
    """x bf16 [M][K], wp = pack_bf16(w) for w [N][K] -> fp32 [M][N] = x . w^T.  With split the
    K-split scratch is allocated here unless a workspace is given; without, no K split."""
    _require_cuda(x, wp)
    assert x.dtype == torch.bfloat16 and x.stride(1) == 1
    M, K = x.shape
    out = torch.empty(M, N, dtype=torch.float32, device=x.device) if out is None else out
    if split and workspace is None:
        need = lib().adt_gemm_bf16_packed_workspace_size(M, N, K)
        workspace = torch.empty(need, dtype=torch.uint8, device=x.device) if need else None
    ws, nbytes = (workspace, workspace.numel()) if split and workspace is not None else (None, 0)
    check(lib().adt_gemm_bf16_packed(_p(x), x.stride(0), _p(wp), M, N, K, _p(out), out.stride(0), _p(ws), nbytes,
                                     _stream()))
    return out


def codebook_knn(codebook: torch.Tensor, k: int) -> torch.Tensor:
    """codebook fp32 [n][dim] -> int32 [n][k]: each code, then its k-1 most cosine-similar codes."""
    _require_cuda(codebook)
    n, dim = codebook.shape
    out = torch.empty(n, k, dtype=torch.int32, device=codebook.device)
    ws = torch.empty(lib().adt_codebook_knn_workspace_size(n), dtype=torch.uint8, device=codebook.device)
    check(lib().adt_codebook_knn(_p(codebook), n, dim, k, _p(out), _p(ws), ws.numel(), _stream()))
    return out


def schedule_next(sched: abi.SchedCfg, left, prev, remaining: int):
    """Host-only schedule: left = (d, k) or None, prev = (a, d) or None."""
    d = C.c_int32()
    k = C.c_int32()
    check(lib().adt_schedule_next(C.byref(sched), 1 if left else 0, left[0] if left else 0, left[1] if left else 0,
                                  1 if prev else 0, prev[0] if prev else 0, prev[1] if prev else 0, remaining,
                                  C.byref(d), C.byref(k)))
    return d.value, k.value


INIT_MODES = {"horizontal": abi.INIT_HORIZONTAL, "vertical": abi.INIT_VERTICAL, "random": abi.INIT_RANDOM,
              "tokenflock": abi.INIT_TOKENFLOCK}
K_CLAMPS = {"always": abi.KCLAMP_ALWAYS, "deep": abi.KCLAMP_DEEP}


def schedule_init(sched: abi.SchedCfg, cell: int, records: dict, n_cells: int):
    """Host-only initial (d~, k~) of the cycle starting at `cell` from records {cell: (d, k)};
    None = no source (the first tree's (d0, k0) without adaptation)."""
    rd = (C.c_int32 * n_cells)()
    rk = (C.c_int32 * n_cells)()
    hr = (C.c_int32 * n_cells)()
    for g, (d, k) in records.items():
        rd[g], rk[g], hr[g] = d, k, 1
    have, d, k = C.c_int32(), C.c_int32(), C.c_int32()
    check(lib().adt_schedule_init(C.byref(sched), cell, n_cells, rd, rk, hr, C.byref(have), C.byref(d), C.byref(k)))
    return (d.value, k.value) if have.value else None


def sched_struct(s, grid_w: int = 0) -> abi.SchedCfg:
    src = abi.ALPHA_POISSON if getattr(s, "alpha_source", "real") == "poisson" else abi.ALPHA_REAL
    return abi.SchedCfg(s.d_lo, s.d_hi, s.k_lo, s.k_hi, s.l_d, s.l_k, s.beta, s.n_budget, s.d0, s.k0, src,
                        INIT_MODES[s.init], grid_w, s.flock_delta, s.fix_d, s.fix_k, K_CLAMPS[s.k_clamp],
                        s.seed & (2 ** 64 - 1))


# ============================================================================ model + session
class DeviceModel:
    """Target model plus draft head on the GPU, weights packed for the GEMM kernels."""

    def __init__(self, cfg, weights: Dict[str, np.ndarray], device="cuda"):
        m = cfg.model
        self.cfg = cfg
        self.dtype = DTYPES[m.dtype]
        self.device = device
        self._keep: List[torch.Tensor] = []
        self.embed = upload(weights["embed"], device)
        self.lm_head = self._pack([weights["lm_head"]], abi.PACK_STACK)
        self.draft_fc = self._pack([weights["draft.fc"]], abi.PACK_STACK)
        qkv_mode = abi.PACK_QKV if self.dtype == abi.BF16 else abi.PACK_STACK
        qkv, o, gu, down = [], [], [], []
        for pre in [f"layer{l}" for l in range(m.n_layers)] + ["draft"]:
            qkv.append(self._pack([weights[pre + ".wq"], weights[pre + ".wk"], weights[pre + ".wv"]], qkv_mode,
                                  m.head_dim))
            o.append(self._pack([weights[pre + ".wo"]], abi.PACK_STACK))
            gu.append(self._pack([weights[pre + ".wg"], weights[pre + ".wu"]], abi.PACK_GATE_UP))
            down.append(self._pack([weights[pre + ".wd"]], abi.PACK_STACK))
        self.qkv, self.o, self.gu, self.down = qkv, o, gu, down
        ptrs = lambda ts: (C.c_void_p * len(ts))(*[t.data_ptr() for t in ts])
        self._arrays = [ptrs(qkv), ptrs(o), ptrs(gu), ptrs(down)]
        desc = abi.ModelDesc(m.n_layers, m.d_model, m.n_heads, m.head_dim, m.ffn, m.vocab, self.dtype, 10000.0, 1e-5,
                             _p(self.embed), _p(self.lm_head), _p(self.draft_fc),
                             C.cast(self._arrays[0], C.POINTER(C.c_void_p)),
                             C.cast(self._arrays[1], C.POINTER(C.c_void_p)),
                             C.cast(self._arrays[2], C.POINTER(C.c_void_p)),
                             C.cast(self._arrays[3], C.POINTER(C.c_void_p)))
        self.handle = C.c_void_p()
        check(lib().adt_model_create(C.byref(desc), C.byref(self.handle)))

    def _pack(self, arrays: Sequence[np.ndarray], mode: int, group: int = 0) -> torch.Tensor:
        srcs = [upload(a, self.device) for a in arrays]
        rows = [int(a.shape[0]) for a in arrays]
        K = int(arrays[0].shape[1])
        nbytes = lib().adt_packed_bytes(sum(rows), K, self.dtype)
        out = torch.empty(nbytes, dtype=torch.uint8, device=self.device)
        sp = (C.c_void_p * len(srcs))(*[s.data_ptr() for s in srcs])
        rw = (C.c_int32 * len(rows))(*rows)
        check(lib().adt_pack_weight(sp, rw, len(srcs), K, mode, group, self.dtype, _p(out), _stream()))
        torch.cuda.current_stream().synchronize()
        return out

    def __del__(self):
        if getattr(self, "handle", None) and _lib_loaded():
            lib().adt_model_destroy(self.handle)
            self.handle = None


def _lib_loaded() -> bool:
    return abi._lib is not None


class DeviceSession:
    """One image decode on the GPU: caches, workspace and the library's session object."""

    def __init__(self, model: DeviceModel, cfg, poisson: Optional[np.ndarray] = None,
                 knn: Optional[torch.Tensor] = None, accept_seed: Optional[int] = None, fixed_tree: bool = False,
                 accept_mode: Optional[str] = None, draft_table: Optional[torch.Tensor] = None,
                 use_graphs: bool = True, caches: Optional[tuple] = None):
        """caches: optional (k_cache, v_cache) views to use as the target caches (a batch
        passes slices of one allocation); otherwise they are allocated here."""
        m = cfg.model
        self.model = model
        self.cfg = cfg
        dev = model.device
        self.s_cap = ((cfg.prefix_len + cfg.n_image + abi.MAX_NODES + 63) // 64) * 64
        tdt = TORCH_DT[model.dtype]
        guided = getattr(cfg, "guidance", None) is not None
        self.nb = 2 if guided else 1
        br = (2,) if guided else ()       # guidance: conditional and unconditional caches
        if caches is not None:
            self.k_cache, self.v_cache = caches
        else:
            self.k_cache = torch.zeros(*br, m.n_layers, m.n_heads, self.s_cap, m.head_dim, dtype=tdt, device=dev)
            self.v_cache = torch.zeros_like(self.k_cache)
        self.dk_cache = torch.zeros(*br, m.n_heads, self.s_cap, m.head_dim, dtype=tdt, device=dev)
        self.dv_cache = torch.zeros_like(self.dk_cache)
        allowed = np.ascontiguousarray(cfg.allowed_table().reshape(-1), dtype=np.int32)
        self._allowed = (C.c_int32 * allowed.size)(*allowed.tolist())
        self._poisson = None
        if poisson is not None:
            self._poisson = (C.c_int32 * len(poisson))(*[int(x) for x in poisson])
        a = cfg.accept
        mode = accept_mode or a.mode
        self.knn = knn
        self.accept = accept_cfg(mode, a.temperature, a.top_k, a.delta, knn, a.knn_k,
                                 cfg.seed if accept_seed is None else accept_seed, children=a.children)
        desc = abi.SessionDesc(cfg.prefix_len, cfg.n_image, self.s_cap, _p(self.k_cache), _p(self.v_cache),
                               _p(self.dk_cache), _p(self.dv_cache),
                               C.cast(self._allowed, C.POINTER(C.c_int32)), sched_struct(cfg.sched, cfg.grid_w), self.accept,
                               C.cast(self._poisson, C.POINTER(C.c_int32)) if self._poisson is not None else None,
                               1 if fixed_tree else 0, _p(draft_table),
                               0 if draft_table is None else draft_table.shape[0], 1 if use_graphs else 0,
                               1 if guided else 0, float(cfg.guidance) if guided else 0.0, None, 0)
        self.draft_table = draft_table
        need = lib().adt_session_workspace_size(model.handle, C.byref(desc))
        if need == 0:
            check(lib().adt_session_create(model.handle, C.byref(desc), C.byref(C.c_void_p())))
        self.workspace = torch.empty(need, dtype=torch.uint8, device=dev)
        desc.workspace = _p(self.workspace)
        desc.workspace_bytes = need
        self._desc = desc
        self.handle = C.c_void_p()
        check(lib().adt_session_create(model.handle, C.byref(desc), C.byref(self.handle)))

    def __del__(self):
        if getattr(self, "handle", None) and _lib_loaded():
            lib().adt_session_destroy(self.handle)
            self.handle = None

    # -- cycle pieces ----------------------------------------------------------------------
    def prefill(self, prefix: np.ndarray, uncond_prefix: Optional[np.ndarray] = None) -> int:
        """prefix: the prompt ids; with guidance also the unconditional prompt (same length)."""
        ids = list(prefix) + (list(uncond_prefix) if self.nb == 2 else [])
        if (self.nb == 2) != (uncond_prefix is not None):
            raise ValueError("an unconditional prompt is needed exactly when the session is guided")
        arr = (C.c_int32 * len(ids))(*[int(x) for x in ids])
        first = C.c_int32()
        check(lib().adt_session_prefill(self.handle, arr, C.byref(first), _stream()))
        return first.value

    def step(self) -> dict:
        out = abi.StepOut()
        check(lib().adt_step(self.handle, C.byref(out), _stream()))
        return _step_dict(out)

    def expand(self, d_hat: int, k_hat: int, n_budget: int) -> int:
        n = C.c_int32()
        check(lib().adt_tree_expand(self.handle, d_hat, k_hat, n_budget, C.byref(n), _stream()))
        return n.value

    def set_tree(self, parent: Sequence[int], token: Sequence[int]) -> None:
        n = len(parent)
        pa = (C.c_int32 * n)(*[int(x) for x in parent])
        to = (C.c_int32 * n)(*[int(x) for x in token])
        check(lib().adt_session_set_tree(self.handle, pa, to, n, _stream()))

    def verify(self) -> None:
        check(lib().adt_verify_forward(self.handle, _stream()))

    def accept_commit(self, d_hat: int, k_hat: int) -> dict:
        out = abi.StepOut()
        check(lib().adt_session_accept_commit(self.handle, d_hat, k_hat, C.byref(out), _stream()))
        return _step_dict(out)

    # -- inspection (views into the session workspace) -------------------------------------
    def view(self) -> abi.SessionView:
        v = abi.SessionView()
        check(lib().adt_session_get_view(self.handle, C.byref(v)))
        return v

    # -- layer-by-layer record (adt_session_set_capture) -------------------------------------
    def set_capture(self, resid_elems: int = 0, xin_bytes: int = 0, meta_elems: int = 0) -> None:
        """Allocates the record buffers and (re)starts recording; resid_elems = 0 stops."""
        dev = self.model.device
        if resid_elems <= 0:
            self._capture = None
            check(lib().adt_session_set_capture(self.handle, None))
            return
        bufs = (torch.empty(resid_elems, dtype=torch.float32, device=dev),
                torch.empty(max(xin_bytes, 16), dtype=torch.uint8, device=dev),
                torch.empty(max(meta_elems, 16), dtype=torch.int32, device=dev))
        cap = abi.Capture(_p(bufs[0]), resid_elems, _p(bufs[1]), xin_bytes, _p(bufs[2]), meta_elems)
        check(lib().adt_session_set_capture(self.handle, C.byref(cap)))
        self._capture = bufs

    def restart_capture(self) -> None:
        """Clears the record, keeping the buffers."""
        r, x, m = self._capture
        cap = abi.Capture(_p(r), r.numel(), _p(x), x.numel(), _p(m), m.numel())
        check(lib().adt_session_set_capture(self.handle, C.byref(cap)))

    def captured(self) -> List[dict]:
        """Every recorded forward since the last (re)start: its record fields, the residual
        snapshots [snapshots][rows][d_model] fp32, the FC input rows (draft forwards), and
        tokens, positions and ancestor masks per node (host arrays)."""
        res, xin, meta = self._capture
        torch.cuda.current_stream().synchronize()
        d = self.cfg.model.d_model
        tdt = TORCH_DT[self.model.dtype]
        out = []
        for i in range(lib().adt_session_capture_count(self.handle)):
            r = abi.CaptureRec()
            check(lib().adt_session_capture_record(self.handle, i, C.byref(r)))
            n, rows = r.nodes, r.rows
            rec = {f: getattr(r, f) for f, _ in abi.CaptureRec._fields_}
            rec["resid"] = res[r.resid_off: r.resid_off + r.snapshots * rows * d].view(r.snapshots, rows, d).cpu()
            if r.draft:
                nb = rows * 2 * d * torch.empty((), dtype=tdt).element_size()
                rec["xin"] = xin[r.xin_off: r.xin_off + nb].view(tdt).view(rows, 2 * d).cpu()
            mt = meta[r.meta_off: r.meta_off + 6 * n].cpu()
            rec["tok"] = mt[:n].numpy().copy()
            rec["pos"] = mt[n: 2 * n].numpy().copy()
            rec["mask"] = mt[2 * n:].numpy().view(np.uint64).reshape(n, 2).copy()
            out.append(rec)
        return out

    def _ws(self, ptr: int, count: int, dtype: torch.dtype) -> torch.Tensor:
        off = ptr - self.workspace.data_ptr()
        nb = count * torch.empty((), dtype=dtype).element_size()
        assert 0 <= off and off + nb <= self.workspace.numel()
        return self.workspace[off: off + nb].view(dtype)

    def tensors(self) -> dict:
        v = self.view()
        m = self.cfg.model
        n = v.n_nodes
        tdt = TORCH_DT[self.model.dtype]
        s = self.cfg.sched
        nb = v.n_branches
        out = {
            "L": v.L, "Ld": v.Ld, "n": n, "step": v.step,
            "logits": self._ws(v.logits, n * m.vocab, torch.float32).view(n, m.vocab),
            "feat": self._ws(v.feat, n * nb * m.d_model, tdt).view(n, nb, m.d_model).squeeze(1),
            "draft_logits": self._ws(v.draft_logits, (1 + (s.d_hi - 1) * s.k_hi) * m.vocab,
                                     torch.float32).view(-1, m.vocab),
            "parent": self._ws(v.parent, n, torch.int32), "token": self._ws(v.token, n, torch.int32),
            "depth": self._ws(v.depth, n, torch.int32), "score": self._ws(v.score, n, torch.float32),
            "mask": self._ws(v.mask, 2 * n, torch.int64).view(n, 2),
            "allowed": self._ws(v.allowed_rows, 2 * n, torch.int32).view(n, 2),
            "path": self._ws(v.path, n, torch.int32), "n_acc": self._ws(v.n_acc, 1, torch.int32),
            "bonus": self._ws(v.bonus, 1, torch.int32),
            "tokens": [v.tokens_host[i] for i in range(v.n_tokens)],
            "logits_range": (v.logits_lo, v.logits_hi),
        }
        if nb == 2:
            out["branch_logits"] = self._ws(v.branch_logits, n * 2 * m.vocab, torch.float32).view(n, 2, m.vocab)
            out["draft_branch_logits"] = self._ws(v.draft_branch_logits, 2 * m.vocab, torch.float32).view(2, m.vocab)
        return out


class DeviceBatch:
    """Several images decoded together: B sessions of one model whose target caches are
    slices of one [B][layers][heads][s_cap][head_dim] allocation, verified by one forward
    per cycle (adt_batch_step)."""

    def __init__(self, model: DeviceModel, cfgs: Sequence, fixed_tree: bool = False):
        m = cfgs[0].model
        B = len(cfgs)
        s_cap = ((cfgs[0].prefix_len + cfgs[0].n_image + abi.MAX_NODES + 63) // 64) * 64
        tdt = TORCH_DT[model.dtype]
        self.k_cache = torch.zeros(B, m.n_layers, m.n_heads, s_cap, m.head_dim, dtype=tdt, device=model.device)
        self.v_cache = torch.zeros_like(self.k_cache)
        self.sessions = [DeviceSession(model, c, fixed_tree=fixed_tree, use_graphs=False,
                                       caches=(self.k_cache[b], self.v_cache[b])) for b, c in enumerate(cfgs)]
        self._handles = (C.c_void_p * B)(*[s.handle.value for s in self.sessions])
        self.handle = None

    def prefill(self, prefixes: Sequence[np.ndarray]) -> List[int]:
        firsts = [s.prefill(p) for s, p in zip(self.sessions, prefixes)]
        B = len(self.sessions)
        need = lib().adt_batch_workspace_size(self._handles, B)
        if need == 0:
            check(lib().adt_batch_create(self._handles, B, None, 0, C.byref(C.c_void_p())))
        self.workspace = torch.empty(need, dtype=torch.uint8, device=self.k_cache.device)
        self.handle = C.c_void_p()
        check(lib().adt_batch_create(self._handles, B, _p(self.workspace), need, C.byref(self.handle)))
        return firsts

    def step(self) -> List[dict]:
        outs = (abi.StepOut * len(self.sessions))()
        check(lib().adt_batch_step(self.handle, outs, _stream()))
        return [_step_dict(o) for o in outs]

    def __del__(self):
        if getattr(self, "handle", None) and _lib_loaded():
            lib().adt_batch_destroy(self.handle)
            self.handle = None


def _step_dict(o: abi.StepOut) -> dict:
    return {"step": o.step, "d_hat": o.d_hat, "k_hat": o.k_hat, "n_nodes": o.n_nodes, "n_accepted": o.n_accepted,
            "n_committed": o.n_committed, "tokens": [o.tokens[i] for i in range(o.n_committed)], "done": o.done}
