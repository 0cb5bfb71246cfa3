"""Seeded synthetic inputs shared by the oracle and the HIP path.

This module only draws random numbers and lays out configuration constants.
It holds none of the method's arithmetic (no norms, attention, scoring,
acceptance or masks): both the oracle and the HIP path take what it returns as
plain inputs.

The paper evaluates on real captions (MS-COCO 2017 val, PartiPrompts) and
ImageNet classes with trained Anole / LlamaGen / Lumina-mGPT weights (Sec. 5.1).
None of those are available, so every model here is a random-init transformer
of the named shape and every prompt is a seeded list of ids; no dataset item is
reproduced.
"""
from __future__ import annotations

import dataclasses
from concurrent.futures import ThreadPoolExecutor
from typing import Dict, List, Optional, Tuple

import numpy as np

CHUNK = 1 << 22          # elements per independently seeded chunk of a tensor
WEIGHT_STD = np.float32(0.02)


@dataclasses.dataclass(frozen=True)
class ModelDims:
    n_layers: int
    d_model: int
    n_heads: int
    head_dim: int
    ffn: int
    vocab: int
    dtype: str            # "f32" or "bf16"

    @property
    def n_params_layer(self) -> int:
        d, f = self.d_model, self.ffn
        return 4 * d * d + 3 * d * f


@dataclasses.dataclass(frozen=True)
class SchedCfg:
    """Tree-shape controls of Sec. 4 (Eq. 2 and the bounds of Sec. 4.2)."""
    d_lo: int
    d_hi: int
    k_lo: int
    k_hi: int
    l_d: int
    l_k: int
    beta: float
    n_budget: int          # draft nodes kept after the top-N rerank (root not counted)
    d0: int                # tree of the first step (no neighbour yet)
    k0: int
    alpha_source: str = "real"   # "real" | "poisson"
    init: str = "horizontal"     # initial (d~, k~): "horizontal" | "vertical" | "random" | "tokenflock"
    flock_delta: int = 2         # TokenFlock radius in grid cells
    fix_d: int = 0               # fixed initial depth (Table V ablations), 0 = none
    fix_k: int = 0               # fixed initial width, 0 = none
    k_clamp: str = "always"      # "always" | "deep": width bounds only when the adapted depth exceeds 1
    seed: int = 0                # key of the Random initialisation


@dataclasses.dataclass(frozen=True)
class AcceptCfg:
    mode: str = "greedy"   # "greedy" | "exact" | "relaxed" | "mss" (stochastic children, Eq. 1 as printed)
    temperature: float = 1.0
    top_k: int = 0         # 0 = untruncated
    delta: float = 0.0
    knn_k: int = 1
    children: int = 0      # mss: children drawn per expanded node


@dataclasses.dataclass(frozen=True)
class DecodeCfg:
    name: str
    model: ModelDims
    seed: int
    prefix_len: int
    prefix_lo: int
    prefix_hi: int
    grid_h: int
    grid_w: int            # tokens per grid row, including a row-end column if any
    img_lo: int            # allowed id range at ordinary image positions
    img_hi: int
    row_end_col: int       # column holding the forced row-end id, or -1
    row_end_id: int
    sched: SchedCfg
    accept: AcceptCfg
    codebook: Optional[Tuple[int, int]] = None   # (entries, dim) for relaxed mode
    guidance: Optional[float] = None   # classifier-free guidance scale (two branches), None = off

    @property
    def n_image(self) -> int:
        return self.grid_h * self.grid_w

    def allowed(self, g: int) -> Tuple[int, int]:
        """Allowed id range [lo, hi) for image cell g (raster order)."""
        if self.row_end_col >= 0:
            if g % self.grid_w == self.row_end_col:
                return (self.row_end_id, self.row_end_id + 1)
        return (self.img_lo, self.img_hi)

    def allowed_table(self) -> np.ndarray:
        t = np.zeros((self.n_image, 2), dtype=np.int32)
        for g in range(self.n_image):
            t[g] = self.allowed(g)
        return t


def _cfg_tiny() -> DecodeCfg:
    m = ModelDims(2, 256, 4, 64, 1024, 1056, "f32")
    return DecodeCfg("tiny", m, seed=0, prefix_len=64, prefix_lo=1024, prefix_hi=1056,
                     grid_h=16, grid_w=16, img_lo=0, img_hi=1024, row_end_col=-1, row_end_id=-1,
                     sched=SchedCfg(1, 4, 1, 4, 1, 1, 1.0, 16, 4, 4),
                     accept=AcceptCfg("greedy"))


def _cfg_llamagen() -> DecodeCfg:
    m = ModelDims(36, 1280, 20, 64, 3584, 16384, "bf16")
    return DecodeCfg("llamagen_xl", m, seed=1, prefix_len=120, prefix_lo=0, prefix_hi=16384,
                     grid_h=32, grid_w=32, img_lo=0, img_hi=16384, row_end_col=-1, row_end_id=-1,
                     sched=SchedCfg(1, 6, 4, 10, 1, 10, 1.0, 60, 5, 10),
                     accept=AcceptCfg("greedy"))


def _cfg_lumina() -> DecodeCfg:
    m = ModelDims(32, 4096, 32, 128, 11008, 65536, "bf16")
    return DecodeCfg("lumina_7b", m, seed=2, prefix_len=64, prefix_lo=0, prefix_hi=65535,
                     grid_h=48, grid_w=49, img_lo=0, img_hi=65535, row_end_col=48, row_end_id=65535,
                     sched=SchedCfg(1, 8, 1, 10, 1, 3, 1.0, 60, 5, 10, alpha_source="poisson"),
                     accept=AcceptCfg("greedy"))


def _cfg_anole(mode: str = "exact") -> DecodeCfg:
    m = ModelDims(32, 4096, 32, 128, 11008, 65536, "bf16")
    return DecodeCfg("anole_7b", m, seed=4, prefix_len=64, prefix_lo=8192, prefix_hi=65536,
                     grid_h=32, grid_w=32, img_lo=0, img_hi=8192, row_end_col=-1, row_end_id=-1,
                     sched=SchedCfg(1, 9, 4, 13, 1, 3, 1.0, 60, 5, 10),
                     accept=AcceptCfg(mode, temperature=1.0, top_k=2000,
                                      delta=0.1 if mode == "relaxed" else 0.0,
                                      knn_k=100 if mode == "relaxed" else 1),
                     codebook=(8192, 256))


CONFIGS = {
    "tiny": _cfg_tiny,
    "llamagen_xl": _cfg_llamagen,
    "lumina_7b": _cfg_lumina,
    "anole_7b": _cfg_anole,
}


def get_config(name: str, **kw) -> DecodeCfg:
    return CONFIGS[name](**kw) if kw else CONFIGS[name]()


def shrink(cfg: DecodeCfg, **model_overrides) -> DecodeCfg:
    """Same decode settings on a smaller model (for fast tests)."""
    m = dataclasses.replace(cfg.model, **model_overrides)
    return dataclasses.replace(cfg, model=m)


# --------------------------------------------------------------------------- weights
# Tensor ids: embedding 0, LM head 1, draft FC 2, draft layer 8..14, target layer l at
# 16 + 8*l + j with j = q, k, v, o, gate, up, down.  Every matrix is [out][in].
LAYER_NAMES = ("wq", "wk", "wv", "wo", "wg", "wu", "wd")


def _layer_shapes(m: ModelDims) -> List[Tuple[int, int]]:
    d, f = m.d_model, m.ffn
    return [(d, d), (d, d), (d, d), (d, d), (f, d), (f, d), (d, f)]


def tensor_table(m: ModelDims) -> List[Tuple[str, int, Tuple[int, int]]]:
    d = m.d_model
    t = [("embed", 0, (m.vocab, d)), ("lm_head", 1, (m.vocab, d)), ("draft.fc", 2, (d, 2 * d))]
    for j, (nm, shp) in enumerate(zip(LAYER_NAMES, _layer_shapes(m))):
        t.append((f"draft.{nm}", 8 + j, shp))
    for l in range(m.n_layers):
        for j, (nm, shp) in enumerate(zip(LAYER_NAMES, _layer_shapes(m))):
            t.append((f"layer{l}.{nm}", 16 + 8 * l + j, shp))
    return t


def _draw_chunk(seed: int, tid: int, c: int, n: int, std: np.float32, bf16: bool) -> np.ndarray:
    x = np.random.default_rng([seed, tid, c]).standard_normal(n, dtype=np.float32)
    x *= std
    if not bf16:
        return x
    # float32 -> bfloat16 bit pattern, round to nearest even (finite inputs only)
    b = x.view(np.uint32)
    t = b >> 16
    t &= 1
    t += 0x7FFF
    b += t
    b >>= 16
    return b.astype(np.uint16)


def draw_tensor(seed: int, tid: int, shape: Tuple[int, ...], bf16: bool,
                std: np.float32 = WEIGHT_STD, pool: Optional[ThreadPoolExecutor] = None) -> np.ndarray:
    """N(0, std^2) tensor; chunk c of the flattened tensor comes from default_rng([seed, tid, c]).

    bf16=True returns uint16 bfloat16 bit patterns, else float32 values."""
    size = int(np.prod(shape))
    nch = (size + CHUNK - 1) // CHUNK
    args = [(seed, tid, c, min(CHUNK, size - c * CHUNK), std, bf16) for c in range(nch)]
    if pool is not None and nch > 1:
        parts = list(pool.map(lambda a: _draw_chunk(*a), args))
    else:
        parts = [_draw_chunk(*a) for a in args]
    return np.concatenate(parts).reshape(shape)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns to float32 (a bit shift)."""
    return (b.astype(np.uint32) << 16).view(np.float32)


def model_weights(cfg: DecodeCfg, threads: int = 8, names: Optional[List[str]] = None) -> Dict[str, np.ndarray]:
    """All weights of the target and the draft head, keyed by name.

    bf16 configs give uint16 bit patterns; f32 configs give float32.  RMSNorm gains
    are 1.0 and are not stored."""
    m = cfg.model
    bf16 = m.dtype == "bf16"
    out: Dict[str, np.ndarray] = {}
    with ThreadPoolExecutor(threads) as pool:
        for name, tid, shape in tensor_table(m):
            if names is not None and name not in names:
                continue
            out[name] = draw_tensor(cfg.seed, tid, shape, bf16, pool=pool)
    return out


def prefix_ids(cfg: DecodeCfg) -> np.ndarray:
    r = np.random.default_rng([cfg.seed, 10_000])
    return r.integers(cfg.prefix_lo, cfg.prefix_hi, size=cfg.prefix_len, dtype=np.int64).astype(np.int32)


def null_prefix_ids(cfg: DecodeCfg) -> np.ndarray:
    """The unconditional prompt of a guided configuration: as long as the prompt, every
    position holding one reserved id (the last id of the prompt range)."""
    return np.full(cfg.prefix_len, cfg.prefix_hi - 1, dtype=np.int32)


def poisson_table(cfg: DecodeCfg) -> np.ndarray:
    """Per-cell acceptance lengths A[g] ~ Poisson(lambda), lambda = 4 on 8x8 blocks whose
    block-row + block-col is even, else 1 (a checkerboard of easy / hard regions)."""
    r = np.random.default_rng([cfg.seed, 7])
    i = np.arange(cfg.grid_h)[:, None] // 8
    j = np.arange(cfg.grid_w)[None, :] // 8
    lam = np.where(((i + j) % 2) == 0, 4.0, 1.0)
    return r.poisson(lam).astype(np.int32).reshape(-1)


def codebook(cfg: DecodeCfg) -> np.ndarray:
    n, dim = cfg.codebook
    return np.random.default_rng([cfg.seed, 20_000]).standard_normal((n, dim), dtype=np.float32)


# --------------------------------------------------------------------------- microbench inputs
@dataclasses.dataclass
class AttnBatch:
    q: np.ndarray          # [B][n_max][H][Dh] bf16 bits
    k: np.ndarray          # [B][H][S_cap][Dh] bf16 bits
    v: np.ndarray
    kv_len: np.ndarray     # [B] committed prefix length L_b
    n_nodes: np.ndarray    # [B] tree rows (root included)
    parent: np.ndarray     # [B][n_max], -1 for the root and for unused rows


def random_parents(rng: np.random.Generator, n: int, max_children: int = 10, max_depth: int = 12) -> np.ndarray:
    """BFS-ordered random tree with n nodes: pop nodes in order, give each node of
    depth < max_depth U{1..max_children} children until the budget is used."""
    parent = np.full(n, -1, dtype=np.int32)
    depth = np.zeros(n, dtype=np.int32)
    nxt, head = 1, 0
    while nxt < n:
        if head >= nxt:        # every open node was at max depth; restart under the root
            head = 0
        if depth[head] < max_depth:
            c = int(rng.integers(1, max_children + 1))
            for _ in range(c):
                if nxt >= n:
                    break
                parent[nxt] = head
                depth[nxt] = depth[head] + 1
                nxt += 1
        head += 1
    return parent


def attn_microbench(B: int, H: int, Dh: int, n: int, seed: int = 3, s_cap: Optional[int] = None,
                    l_lo: int = 512, l_hi: int = 2400, vary_n: bool = False) -> AttnBatch:
    """Batch of independent sequences with random trees over bf16 caches, entries ~N(0,1)."""
    rng = np.random.default_rng([seed, n, B, H, Dh])
    kv_len = rng.integers(l_lo, l_hi + 1, size=B).astype(np.int32)
    n_nodes = (rng.integers(1, n + 1, size=B) if vary_n else np.full(B, n)).astype(np.int32)
    if s_cap is None:
        s_cap = int(kv_len.max()) + n
    parent = np.full((B, n), -1, dtype=np.int32)
    for b in range(B):
        parent[b, :n_nodes[b]] = random_parents(rng, int(n_nodes[b]))
    q = draw_tensor(seed, 1_000 + n, (B, n, H, Dh), True, std=np.float32(1.0))
    k = draw_tensor(seed, 2_000 + n, (B, H, s_cap, Dh), True, std=np.float32(1.0))
    v = draw_tensor(seed, 3_000 + n, (B, H, s_cap, Dh), True, std=np.float32(1.0))
    return AttnBatch(q, k, v, kv_len, n_nodes, parent)


def compaction_paths(rng: np.random.Generator, n_nodes: np.ndarray, a_max: int = 12) -> Tuple[np.ndarray, np.ndarray]:
    """Accepted paths for compaction: a ~ U{1..min(a_max, n-1)}, sorted distinct
    node indices in [1, n).  Returns (path [B][a_max+1] with path[0] = 0, a [B])."""
    B = len(n_nodes)
    path = np.zeros((B, a_max + 1), dtype=np.int32)
    a = np.zeros(B, dtype=np.int32)
    for b in range(B):
        n = int(n_nodes[b])
        if n < 2:
            continue
        ab = int(rng.integers(1, min(a_max, n - 1) + 1))
        sel = np.sort(rng.choice(np.arange(1, n), size=ab, replace=False))
        path[b, 1:ab + 1] = sel
        a[b] = ab
    return path, a


def random_knn_table(rows: int, k: int, seed: int = 0) -> np.ndarray:
    """A neighbour table for acceptance tests: row x lists x first, then k-1 other ids in a
    seeded random order (no similarity computation)."""
    rng = np.random.default_rng([seed, 30_000])
    out = np.zeros((rows, k), dtype=np.int32)
    for x in range(rows):
        others = rng.choice(rows - 1, size=k - 1, replace=False)
        others = others + (others >= x)
        out[x, 0] = x
        out[x, 1:] = others
    return out
