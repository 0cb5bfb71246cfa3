"""Whole-cycle pins of the oracle: the method is lossless in greedy mode (Sec. 5.1), so
tree decoding must reproduce the target's plain greedy AR output token for token."""
import dataclasses

import numpy as np
import pytest

import synth
from oracle.decode import Decoder, ar_decode
from oracle.model import OracleModel


@pytest.fixture(scope="module")
def tiny():
    cfg = synth.get_config("tiny")
    w = synth.model_weights(cfg)
    model = OracleModel(cfg, w)
    pre = synth.prefix_ids(cfg)
    ar, ar_rows = ar_decode(cfg, model, pre)
    return cfg, w, model, pre, ar, ar_rows


def _plant_draft(model, full_seq, V, rng_seed=0):
    """Replace the draft logits: a row whose token matches the AR sequence at its position
    proposes the AR continuation (plus noise), any other row proposes noise.  Only the draft
    quality changes; whatever the draft proposes, the committed tokens must equal AR."""
    real = model.draft_rows

    def planted(tokens, parent_feat, pos, slots, key_slots, cache):
        lg, fd = real(tokens, parent_feat, pos, slots, key_slots, cache)
        out = np.random.default_rng([rng_seed, int(pos[0]), len(pos)]).standard_normal(lg.shape)
        for r, (t, p) in enumerate(zip(tokens, pos)):
            if p + 1 < len(full_seq) and int(t) == full_seq[p]:
                out[r, full_seq[p + 1]] += 8.0
        return out, fd
    model.draft_rows = planted
    return real


def test_greedy_tree_decode_equals_ar_random_draft(tiny):
    cfg, w, model, pre, ar, _ = tiny
    dec = Decoder(cfg, model, pre)
    dec.prefill()
    infos = dec.run()
    assert dec.tokens[len(pre):] == ar
    assert sum(len(i.committed) for i in infos) + 1 == cfg.n_image


def test_greedy_tree_decode_equals_ar_planted_draft(tiny):
    cfg, w, _, pre, ar, _ = tiny
    model = OracleModel(cfg, w)
    full = list(pre) + list(ar)
    _plant_draft(model, full, cfg.model.vocab)
    dec = Decoder(cfg, model, pre)
    dec.prefill()
    infos = dec.run()
    assert dec.tokens[len(pre):] == ar
    acc = [len(i.path) for i in infos]
    assert max(acc) == cfg.sched.d_hi and np.mean(acc) > 2.0       # long paths were accepted
    # positive trees deepen and narrow (Eq. 2): depth reaches its maximum
    assert max(i.d_hat for i in infos) == cfg.sched.d_hi and min(i.k_hat for i in infos) == cfg.sched.k_lo
    for i in infos:
        assert len(i.path) <= i.d_hat and i.tree.n - 1 <= cfg.sched.n_budget


def test_root_logits_equal_ar_logits(tiny):
    cfg, w, model, pre, ar, ar_rows = tiny
    dec = Decoder(cfg, model, pre)
    dec.prefill()
    infos = dec.run(5)
    k = 0
    for info in infos:
        j = len(dec.tokens[: info.L_before + 1]) - len(pre) - 1       # AR row predicting the root's successor
        np.testing.assert_allclose(info.logits[0], ar_rows[j], rtol=1e-10, atol=1e-10)
        k += 1
    assert k == 5


def test_depth_one_width_one_is_ar(tiny):
    cfg, w, model, pre, ar, _ = tiny
    c1 = dataclasses.replace(cfg, sched=dataclasses.replace(cfg.sched, d_lo=1, d_hi=1, k_lo=1, k_hi=1, d0=1, k0=1))
    dec = Decoder(c1, model, pre)
    dec.prefill()
    infos = dec.run(40)
    assert all(i.tree.n == 2 and i.d_hat == 1 and i.k_hat == 1 for i in infos)
    assert dec.tokens[len(pre):] == ar[: len(dec.tokens) - len(pre)]


def test_compacted_cache_equals_ar_cache(tiny):
    cfg, w, _, pre, ar, _ = tiny
    model = OracleModel(cfg, w)
    full = list(pre) + list(ar)
    _plant_draft(model, full, cfg.model.vocab)
    dec = Decoder(cfg, model, pre)
    dec.prefill()
    dec.run(12)
    ref = Decoder(cfg, OracleModel(cfg, w), pre)
    P = len(pre)
    pos = list(range(dec.L))
    ref.model.target_rows(full[: dec.L], pos, pos, [list(range(p + 1)) for p in pos], ref.tcache)
    np.testing.assert_allclose(dec.tcache.k[:, :, : dec.L], ref.tcache.k[:, :, : dec.L], rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dec.tcache.v[:, :, : dec.L], ref.tcache.v[:, :, : dec.L], rtol=1e-10, atol=1e-12)


def test_bf16_rounding_points_bound_error():
    """A bf16-shaped model: the oracle with storage rounding stays within the bf16 tolerance
    of the same model evaluated without any rounding."""
    cfg = synth.shrink(synth.get_config("llamagen_xl"), n_layers=2, d_model=256, n_heads=4, ffn=512, vocab=512)
    cfg = dataclasses.replace(cfg, prefix_len=16, img_hi=512, prefix_hi=512)
    w = synth.model_weights(cfg)
    m_r = OracleModel(cfg, w)
    m_x = OracleModel(cfg, w)
    m_x.rnd = lambda x: x
    pre = synth.prefix_ids(cfg)
    pos = list(range(len(pre)))
    causal = [list(range(r + 1)) for r in pos]
    lr, _ = m_r.target_rows(pre, pos, pos, causal, m_r.new_caches(64)[0])
    lx, _ = m_x.target_rows(pre, pos, pos, causal, m_x.new_caches(64)[0])
    assert np.all(np.abs(lr - lx) <= 2e-2 + 1e-2 * np.abs(lx))
    assert np.abs(lr - lx).max() > 0


# ---------------------------------------------------------------- classifier-free guidance
# Sec. 3.1: p and q are both computed with CFG (conditional and unconditional branches per
# position, Fig. 5 caption); the combination is l_u + s (l_c - l_u) on logits.
def _guided(cfg, s):
    return dataclasses.replace(cfg, guidance=s)


@pytest.mark.parametrize("planted", [False, True])
def test_guided_tree_decode_equals_guided_ar(tiny, planted):
    cfg0, w, _, pre, _, _ = tiny
    cfg = _guided(cfg0, 3.0)
    null = synth.null_prefix_ids(cfg)
    model = OracleModel(cfg, w)
    ar, _ = ar_decode(cfg, model, pre, uncond_prefix=null)
    assert ar != tiny[4]                          # guidance changes the image
    if planted:
        _plant_draft(model, list(pre) + list(ar), cfg.model.vocab)
    dec = Decoder(cfg, model, pre, uncond_prefix=null)
    dec.prefill()
    infos = dec.run()
    assert dec.tokens[len(pre):] == ar
    if planted:
        assert np.mean([len(i.path) for i in infos]) > 2.0


def test_guidance_scale_one_and_zero_reduce_to_one_branch(tiny):
    """s = 1 gives the conditional model's logits, s = 0 the unconditional one's: the guided
    decode then equals a plain decode with that branch's prompt, cycle for cycle."""
    cfg0, w, model, pre, _, _ = tiny
    null = synth.null_prefix_ids(cfg0)
    for s, prompt in ((1.0, pre), (0.0, null)):
        g = Decoder(_guided(cfg0, s), model, pre, uncond_prefix=null)
        p = Decoder(cfg0, model, prompt)
        assert g.prefill() == p.prefill()
        np.testing.assert_allclose(g.prefill_logits, p.prefill_logits, rtol=1e-12, atol=1e-12)
        for _ in range(12):
            gi, pi = g.step(), p.step()
            assert (gi.d_hat, gi.k_hat, gi.committed) == (pi.d_hat, pi.k_hat, pi.committed)
            assert gi.tree.token.tolist() == pi.tree.token.tolist()
            np.testing.assert_allclose(gi.logits, pi.logits, rtol=1e-12, atol=1e-12)
            np.testing.assert_allclose(gi.draft_root_logits, pi.draft_root_logits, rtol=1e-12, atol=1e-12)
