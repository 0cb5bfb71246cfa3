"""Pins of the oracle's elementwise pieces against library routines and closed forms."""
import json
import os

import numpy as np
import pytest
import torch

from oracle.numerics import bf16_round, draw_below, philox4x32_10, rmsnorm, rope, silu, uniform_u64

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def test_bf16_round_matches_torch_cast():
    x = np.random.default_rng(0).standard_normal(100_000).astype(np.float32) * 3.0
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(bf16_round(x.astype(np.float64)), ref)


def test_bf16_round_ties_to_even():
    assert bf16_round(1.0 + 2.0 ** -8) == 1.0                     # halfway, even neighbour is 1.0
    assert bf16_round(1.0 + 3 * 2.0 ** -8) == 1.0 + 2.0 ** -6     # halfway, even neighbour above
    assert bf16_round(-(1.0 + 2.0 ** -8 + 2.0 ** -20)) == -(1.0 + 2.0 ** -7)


def test_rmsnorm_closed_form_and_torch():
    x = np.random.default_rng(1).standard_normal((7, 33))
    y = rmsnorm(x, 1e-5)
    ms = np.mean(x * x, axis=1)
    assert np.allclose(np.mean(y * y, axis=1), ms / (ms + 1e-5), rtol=1e-13)
    ref = torch.nn.functional.rms_norm(torch.from_numpy(x), (33,), eps=1e-5).numpy()
    assert np.allclose(y, ref, rtol=1e-12, atol=1e-14)


def test_silu_matches_torch():
    x = np.linspace(-30, 30, 1001)
    assert np.allclose(silu(x), torch.nn.functional.silu(torch.from_numpy(x)).numpy(), rtol=1e-13, atol=1e-15)


def test_rope_is_complex_rotation():
    """Pair (i, i + Dh/2) of rotate-half RoPE is the complex number x_i + j x_{i+Dh/2}
    multiplied by exp(j * pos * theta^(-2i/Dh))."""
    rng = np.random.default_rng(2)
    x = rng.standard_normal((5, 3, 8))
    pos = np.array([0, 1, 7, 300, 2399])
    y = rope(x, pos)
    z = x[..., :4] + 1j * x[..., 4:]
    freq = 10000.0 ** (-np.arange(4) * 2 / 8)
    zr = z * np.exp(1j * pos[:, None, None] * freq[None, None, :])
    assert np.allclose(y[..., :4], zr.real, atol=1e-12) and np.allclose(y[..., 4:], zr.imag, atol=1e-12)


def test_rope_identity_norm_and_relative_position():
    rng = np.random.default_rng(3)
    q = rng.standard_normal((1, 2, 64))
    k = rng.standard_normal((1, 2, 64))
    assert np.allclose(rope(q, [0]), q)
    assert np.allclose(np.linalg.norm(rope(q, [123]), axis=-1), np.linalg.norm(q, axis=-1))
    d1 = np.sum(rope(q, [40]) * rope(k, [17]), axis=-1)
    d2 = np.sum(rope(q, [40 + 555]) * rope(k, [17 + 555]), axis=-1)
    assert np.allclose(d1, d2, atol=1e-10)


def test_philox_known_answers():
    g = json.load(open(os.path.join(GOLD, "philox4x32_10_kat.json")))
    for v in g["vectors"]:
        out = philox4x32_10([int(x, 16) for x in v["ctr"]], [int(x, 16) for x in v["key"]])
        assert ["%08x" % o for o in out] == v["out"]


def test_draw_below_is_uniform():
    """floor(U * W / 2^64) over Philox words: every residue class of W = 6 equally likely."""
    W = 6
    counts = np.zeros(W)
    for t in range(60_000):
        counts[draw_below(uniform_u64(7, t, 3, 1), W)] += 1
    exp = 60_000 / W
    chi2 = float(np.sum((counts - exp) ** 2 / exp))
    assert chi2 < 25.0            # 5 dof, p ~ 1e-4
    assert draw_below(2 ** 64 - 1, W) == W - 1 and draw_below(0, W) == 0
