"""Target transformer and EAGLE-style draft head of the oracle.

The paper's target model is an AR transformer over image tokens (Sec. 3.1) and its
draft model follows the EAGLE design: the token embedding is concatenated with the
parent's intermediate feature and passed through an FC layer and one decoder layer
(Sec. 4.2 and the caption of Fig. 5).  The layer itself is a plain pre-norm
decoder: RMSNorm, RoPE, multi-head attention, SwiGLU FFN, no biases, untied LM
head; the draft head reuses the target's embedding and LM head.

Test infrastructure only; see the package docstring.
"""
from __future__ import annotations

from typing import Dict, Optional, Sequence

import numpy as np

from synth import DecodeCfg, bf16_bits_to_f32
from .attention import attend_rows
from .numerics import bf16_round, rmsnorm, rope, silu


class KVCache:
    """K and V of one stack of layers: [layers][H][S_cap][Dh] float64."""

    def __init__(self, layers: int, H: int, s_cap: int, Dh: int):
        self.k = np.zeros((layers, H, s_cap, Dh), dtype=np.float64)
        self.v = np.zeros((layers, H, s_cap, Dh), dtype=np.float64)


class OracleModel:
    def __init__(self, cfg: DecodeCfg, weights: Dict[str, np.ndarray], cache_f64: Optional[bool] = None):
        self.cfg = cfg
        self.m = cfg.model
        self.bf16 = self.m.dtype == "bf16"
        self.raw = weights
        total = sum(w.size for w in weights.values())
        self.cache_f64 = (total < 1_200_000_000) if cache_f64 is None else cache_f64
        self._f64: Dict[str, np.ndarray] = {}
        self.scale = 1.0 / np.sqrt(self.m.head_dim)
        self.trace: Optional[Dict[str, np.ndarray]] = None   # set to {} to keep per-layer values

    # -- weights -------------------------------------------------------------------------
    def w(self, name: str) -> np.ndarray:
        if name in self._f64:
            return self._f64[name]
        raw = self.raw[name]
        x = (bf16_bits_to_f32(raw) if raw.dtype == np.uint16 else raw).astype(np.float64)
        if self.cache_f64:
            self._f64[name] = x
        return x

    def rnd(self, x: np.ndarray) -> np.ndarray:
        """Storage rounding of a bf16 model; identity for f32 models."""
        return bf16_round(x) if self.bf16 else x

    def normed_input(self, h: np.ndarray) -> np.ndarray:
        """Input of a layer's projections: the RMSNorm of the residual copy kept in storage
        precision (a bf16 model stores the residual rows, not their norm, and the scale is
        applied in full precision)."""
        return rmsnorm(self.rnd(h))

    def embed_rows(self, tokens: Sequence[int]) -> np.ndarray:
        return self.w("embed")[np.asarray(tokens, dtype=np.int64)]

    # -- one decoder layer over a set of rows ---------------------------------------------
    def attn_block(self, pre: str, h: np.ndarray, pos: Sequence[int], slots: Sequence[int],
                   key_slots: Sequence[Sequence[int]], cache: KVCache, li: int):
        """First half of a pre-norm layer: h + Attn(RMSNorm(h)) W_o.  Row r sits at position
        pos[r]; its K/V are written to cache slot slots[r] before attention, and it attends to
        key_slots[r].  Returns (new residual, q, o)."""
        m = self.m
        rows = h.shape[0]
        H, Dh = m.n_heads, m.head_dim
        a = self.normed_input(h)
        q = (a @ self.w(pre + ".wq").T).reshape(rows, H, Dh)
        k = (a @ self.w(pre + ".wk").T).reshape(rows, H, Dh)
        v = (a @ self.w(pre + ".wv").T).reshape(rows, H, Dh)
        q = self.rnd(rope(q, pos))
        k = self.rnd(rope(k, pos))
        v = self.rnd(v)
        sl = np.asarray(slots, dtype=np.int64)
        cache.k[li][:, sl, :] = k.transpose(1, 0, 2)
        cache.v[li][:, sl, :] = v.transpose(1, 0, 2)
        o = self.rnd(attend_rows(q, cache.k[li], cache.v[li], key_slots, self.scale))
        return h + o.reshape(rows, H * Dh) @ self.w(pre + ".wo").T, q, o

    def mlp_block(self, pre: str, h: np.ndarray):
        """Second half: h + SwiGLU(RMSNorm(h)) W_down.  Returns (new residual, b, s)."""
        b = self.normed_input(h)
        s = self.rnd(silu(b @ self.w(pre + ".wg").T) * (b @ self.w(pre + ".wu").T))
        return h + s @ self.w(pre + ".wd").T, b, s

    def layer(self, pre: str, h: np.ndarray, pos: Sequence[int], slots: Sequence[int],
              key_slots: Sequence[Sequence[int]], cache: KVCache, li: int) -> np.ndarray:
        """h: [rows][d] residual stream through both halves of the layer."""
        rows = h.shape[0]
        h_attn, q, o = self.attn_block(pre, h, pos, slots, key_slots, cache, li)
        out, b, s = self.mlp_block(pre, h_attn)
        if self.trace is not None:
            self.trace.update({pre + ".q": q.reshape(rows, -1), pre + ".o": o.reshape(rows, -1),
                               pre + ".h_attn": h_attn, pre + ".b": b, pre + ".s": s, pre + ".h": out})
        return out

    # -- full forwards ---------------------------------------------------------------------
    def target_rows(self, tokens, pos, slots, key_slots, cache: KVCache):
        """Target forward of a set of rows.  Returns (logits [rows][V], features f [rows][d]),
        f being the final-norm output that feeds the LM head (and the draft head)."""
        h = self.embed_rows(tokens)
        for li in range(self.m.n_layers):
            h = self.layer(f"layer{li}", h, pos, slots, key_slots, cache, li)
        f = self.rnd(rmsnorm(h))
        return f @ self.w("lm_head").T, f

    def draft_rows(self, tokens, parent_feat: np.ndarray, pos, slots, key_slots, cache: KVCache):
        """Draft-head forward: FC over [embedding ; parent feature], one decoder layer, the
        head's own final norm, then the target's LM head.  Returns (logits, draft features)."""
        x = np.concatenate([self.embed_rows(tokens), parent_feat], axis=1)
        h = x @ self.w("draft.fc").T
        h = self.layer("draft", h, pos, slots, key_slots, cache, 0)
        f = self.rnd(rmsnorm(h))
        return f @ self.w("lm_head").T, f

    def new_caches(self, s_cap: int):
        m = self.m
        return KVCache(m.n_layers, m.n_heads, s_cap, m.head_dim), KVCache(1, m.n_heads, s_cap, m.head_dim)
