"""Independent pin of the oracle's transformer (target decoder stack, LM head, draft head).

The reference here is written separately from ``oracle/model.py``: whole sequences at once
in torch float64, ``F.rms_norm``, RoPE as a complex multiplication of the pairs
(i, i + Dh/2), ``F.scaled_dot_product_attention`` with an explicit boolean key mask,
``F.silu``, and ``F.linear`` for every projection.  It follows the architecture the paper
implies (Sec. 3.1: an AR transformer over image tokens; Sec. 4.2 and the caption of Fig. 5:
an EAGLE-style draft head that feeds the concatenation of the token embedding and the
parent's feature through an FC layer and one decoder layer, then the target's LM head), with
the readings the oracle states (pre-norm layers, RMSNorm with unit gain, rotate-half RoPE,
SwiGLU, no biases, untied LM head).

The oracle is evaluated with bf16 storage rounding switched off (f32 model configurations),
so the two must agree to float64 rounding.  A second group of tests plants the plausible
mistakes (gate and up swapped, a norm in the wrong place, a residual added at the wrong
point, the draft FC inputs in the other order, a tied LM head) in a copy of the oracle's
layer and checks that the pin rejects each of them.
"""
import dataclasses

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import synth
from oracle.attention import tree_key_slots
from oracle.model import KVCache, OracleModel
from oracle.numerics import rmsnorm, rope, silu
from oracle.tree import ancestors_and_self

EPS = 1e-5
THETA = 10000.0


# ----------------------------------------------------------------------------- the reference
def _tw(weights, name):
    w = weights[name]
    if w.dtype == np.uint16:
        w = synth.bf16_bits_to_f32(w)
    return torch.from_numpy(np.asarray(w, dtype=np.float64))


def _rotary(x, pos):
    """x [T][H][Dh]; pair (i, i + Dh/2) is the complex number x_i + j x_{i+Dh/2}, turned by
    pos * THETA^(-2i/Dh)."""
    half = x.shape[-1] // 2
    z = torch.complex(x[..., :half], x[..., half:])
    freq = THETA ** (-2.0 * torch.arange(half, dtype=torch.float64) / x.shape[-1])
    ang = torch.as_tensor(pos, dtype=torch.float64)[:, None, None] * freq
    z = z * torch.polar(torch.ones_like(ang), ang)
    return torch.cat([z.real, z.imag], dim=-1)


def ref_layer(weights, pre, x, pos, allowed, H, Dh):
    """One pre-norm decoder layer over a whole sequence.  allowed[i][j]: query i sees key j."""
    T, d = x.shape
    a = F.rms_norm(x, (d,), eps=EPS)
    q = _rotary(F.linear(a, _tw(weights, pre + ".wq")).view(T, H, Dh), pos)
    k = _rotary(F.linear(a, _tw(weights, pre + ".wk")).view(T, H, Dh), pos)
    v = F.linear(a, _tw(weights, pre + ".wv")).view(T, H, Dh)
    o = F.scaled_dot_product_attention(q.transpose(0, 1), k.transpose(0, 1), v.transpose(0, 1),
                                       attn_mask=torch.as_tensor(allowed), scale=Dh ** -0.5)
    x = x + F.linear(o.transpose(0, 1).reshape(T, d), _tw(weights, pre + ".wo"))
    b = F.rms_norm(x, (d,), eps=EPS)
    gate = F.silu(F.linear(b, _tw(weights, pre + ".wg")))
    up = F.linear(b, _tw(weights, pre + ".wu"))
    return x + F.linear(gate * up, _tw(weights, pre + ".wd"))


def ref_target(weights, m, tokens, pos, allowed):
    x = _tw(weights, "embed")[torch.as_tensor(tokens)]
    for li in range(m.n_layers):
        x = ref_layer(weights, f"layer{li}", x, pos, allowed, m.n_heads, m.head_dim)
    f = F.rms_norm(x, (m.d_model,), eps=EPS)
    return F.linear(f, _tw(weights, "lm_head")).numpy(), f.numpy()


def ref_draft(weights, m, tokens, parent_feat, pos, allowed):
    e = _tw(weights, "embed")[torch.as_tensor(tokens)]
    x = F.linear(torch.cat([e, torch.from_numpy(parent_feat)], dim=1), _tw(weights, "draft.fc"))
    x = ref_layer(weights, "draft", x, pos, allowed, m.n_heads, m.head_dim)
    f = F.rms_norm(x, (m.d_model,), eps=EPS)
    return F.linear(f, _tw(weights, "lm_head")).numpy(), f.numpy()


# ----------------------------------------------------------------------------- shapes
def _cfgs():
    tiny = synth.get_config("tiny")
    # a LlamaGen-like shape shrunk, with 128-wide heads and bf16-drawn weights evaluated
    # without storage rounding (the model dtype says f32)
    wide = synth.shrink(synth.get_config("lumina_7b"), n_layers=3, d_model=256, n_heads=2, head_dim=128, ffn=384,
                        vocab=640, dtype="f32")
    wide = dataclasses.replace(wide, prefix_lo=0, prefix_hi=640, img_hi=639, row_end_id=639)
    return {"tiny": tiny, "wide_heads": wide}


CFGS = _cfgs()


@pytest.fixture(scope="module", params=list(CFGS))
def setup(request):
    cfg = CFGS[request.param]
    w = synth.model_weights(cfg, threads=4)
    # bf16-drawn weights for the second shape: the bits are exact in float64 either way
    if request.param == "wide_heads":
        w = {k: synth.draw_tensor(cfg.seed, i, v.shape, True) for i, (k, v) in enumerate(sorted(w.items()))}
    return cfg, w


def _close(a, b, what):
    err = float(np.max(np.abs(np.asarray(a) - np.asarray(b))))
    scale = float(np.max(np.abs(np.asarray(b))))
    assert err <= 1e-12 * max(1.0, scale), f"{what}: max |diff| {err:.3e} (scale {scale:.3g})"


def _causal(T):
    return np.tril(np.ones((T, T), dtype=bool))


# ----------------------------------------------------------------------------- pins
def test_target_forward_matches_reference(setup):
    """A causal sequence through OracleModel.target_rows (row by row, through its cache)
    equals the whole-sequence reference: every layer's output, the final features, the
    logits."""
    cfg, w = setup
    m = cfg.model
    rng = np.random.default_rng(11)
    T = 23
    toks = rng.integers(0, m.vocab, T)
    pos = np.arange(T) + 5                       # positions need not start at 0
    om = OracleModel(cfg, w)
    om.trace = {}
    tc, _ = om.new_caches(64)
    slots = list(range(T))
    logits, f = om.target_rows(toks, pos, slots, [list(range(r + 1)) for r in range(T)], tc)
    rl, rf = ref_target(w, m, toks, pos, _causal(T))
    _close(f, rf, "features")
    _close(logits, rl, "logits")
    # per layer: the oracle's traced residual after each layer equals the reference's
    x = _tw(w, "embed")[torch.as_tensor(toks)]
    for li in range(m.n_layers):
        x = ref_layer(w, f"layer{li}", x, pos, _causal(T), m.n_heads, m.head_dim)
    _close(om.trace[f"layer{m.n_layers - 1}.h"], x.numpy(), "last layer residual")


def test_target_tree_rows_match_reference_on_paths(setup):
    """Tree rows (prefix + each node's ancestors under the tree mask) equal the reference run
    densely on prefix + root-to-node path, node by node (brute force)."""
    cfg, w = setup
    m = cfg.model
    rng = np.random.default_rng(12)
    Lp = 9
    prefix = rng.integers(0, m.vocab, Lp)
    parent = np.array([-1, 0, 0, 1, 1, 2, 3, 3, 6], dtype=np.int32)
    ttok = rng.integers(0, m.vocab, len(parent))
    depth = np.array([len(a) - 1 for a in ancestors_and_self(parent)])
    om = OracleModel(cfg, w)
    tc, _ = om.new_caches(64)
    om.target_rows(prefix, np.arange(Lp), list(range(Lp)), [list(range(r + 1)) for r in range(Lp)], tc)
    anc = ancestors_and_self(parent)
    logits, f = om.target_rows(ttok, Lp + depth, [Lp + i for i in range(len(parent))], tree_key_slots(Lp, anc), tc)
    for i in range(len(parent)):
        seq = np.concatenate([prefix, ttok[anc[i]]])
        rl, rf = ref_target(w, m, seq, np.arange(len(seq)), _causal(len(seq)))
        _close(f[i], rf[-1], f"tree node {i} feature")
        _close(logits[i], rl[-1], f"tree node {i} logits")


def test_draft_head_matches_reference(setup):
    """OracleModel.draft_rows: FC over [embedding ; parent feature], one decoder layer of the
    target's shape, its own final norm and the target's LM head."""
    cfg, w = setup
    m = cfg.model
    rng = np.random.default_rng(13)
    T = 11
    toks = rng.integers(0, m.vocab, T)
    par = rng.standard_normal((T, m.d_model))
    om = OracleModel(cfg, w)
    _, dc = om.new_caches(64)
    logits, f = om.draft_rows(toks, par, np.arange(T), list(range(T)), [list(range(r + 1)) for r in range(T)], dc)
    rl, rf = ref_draft(w, m, toks, par, np.arange(T), _causal(T))
    _close(f, rf, "draft features")
    _close(logits, rl, "draft logits")


# ----------------------------------------------------------------------------- planted mistakes
def _mutant_layer(kind):
    """A copy of the oracle's layer arithmetic with one planted mistake."""

    def layer(self, pre, h, pos, slots, key_slots, cache: KVCache, li):
        from oracle.attention import attend_rows
        m = self.m
        rows = h.shape[0]
        H, Dh = m.n_heads, m.head_dim
        a = rmsnorm(h)
        q = (a @ self.w(pre + ".wq").T).reshape(rows, H, Dh)
        k = (a @ self.w(pre + ".wk").T).reshape(rows, H, Dh)
        v = (a @ self.w(pre + ".wv").T).reshape(rows, H, Dh)
        q, k = rope(q, pos), rope(k, pos)
        sl = np.asarray(slots)
        cache.k[li][:, sl, :] = k.transpose(1, 0, 2)
        cache.v[li][:, sl, :] = v.transpose(1, 0, 2)
        o = attend_rows(q, cache.k[li], cache.v[li], key_slots, self.scale).reshape(rows, H * Dh)
        attn = o @ self.w(pre + ".wo").T
        h2 = attn if kind == "attn_residual_dropped" else h + attn
        b = rmsnorm(h if kind == "mlp_norm_of_layer_input" else h2)
        g, u = (".wu", ".wg") if kind == "gate_up_swapped" else (".wg", ".wu")
        s = silu(b @ self.w(pre + g).T) * (b @ self.w(pre + u).T)
        base = h if kind == "mlp_residual_on_layer_input" else h2
        return base + s @ self.w(pre + ".wd").T

    return layer


@pytest.mark.parametrize("kind", ["gate_up_swapped", "mlp_norm_of_layer_input", "attn_residual_dropped",
                                  "mlp_residual_on_layer_input", "draft_fc_inputs_swapped", "lm_head_tied",
                                  "sanity_unchanged"])
def test_pin_rejects_planted_mistakes(kind, monkeypatch):
    cfg = CFGS["tiny"]
    w = synth.model_weights(cfg, threads=4)
    m = cfg.model
    om = OracleModel(cfg, w)
    if kind in ("gate_up_swapped", "mlp_norm_of_layer_input", "attn_residual_dropped",
                "mlp_residual_on_layer_input"):
        monkeypatch.setattr(OracleModel, "layer", _mutant_layer(kind))
    elif kind == "sanity_unchanged":
        monkeypatch.setattr(OracleModel, "layer", _mutant_layer("none"))
    elif kind == "lm_head_tied":
        om.raw = dict(w, lm_head=w["embed"])
    rng = np.random.default_rng(14)
    T = 7
    toks = rng.integers(0, m.vocab, T)
    par = rng.standard_normal((T, m.d_model))
    keys = [list(range(r + 1)) for r in range(T)]
    tc, dc = om.new_caches(32)
    if kind == "draft_fc_inputs_swapped":
        x = np.concatenate([par, om.embed_rows(toks)], axis=1) @ om.w("draft.fc").T
        got = om.layer("draft", x, np.arange(T), list(range(T)), keys, dc, 0)
        f = rmsnorm(got)
        got_logits = f @ om.w("lm_head").T
    else:
        got_logits, _ = om.draft_rows(toks, par, np.arange(T), list(range(T)), keys, dc)
    rl, _ = ref_draft(w, m, toks, par, np.arange(T), _causal(T))
    tl, _ = om.target_rows(toks, np.arange(T), list(range(T)), keys, tc)
    rt, _ = ref_target(w, m, toks, np.arange(T), _causal(T))
    if kind == "sanity_unchanged":
        _close(got_logits, rl, "draft logits")
        _close(tl, rt, "target logits")
        return
    with pytest.raises(AssertionError):
        _close(got_logits, rl, "draft logits")
        _close(tl, rt, "target logits")
