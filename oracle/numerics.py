"""Elementwise building blocks of the oracle (float64 NumPy).

Test infrastructure only; see the package docstring.
"""
from __future__ import annotations

import numpy as np

MASK32 = 0xFFFFFFFF


def bf16_round(x) -> np.ndarray:
    """Nearest bfloat16 value (8 significant bits), ties to even, returned as float64.

    Writes x = m * 2**e with 0.5 <= |m| < 1 and rounds m * 2**8 to an integer.
    Values below the bfloat16 normal range are not expected here."""
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)
    return np.ldexp(np.round(np.ldexp(m, 8)), e - 8)


def rmsnorm(x: np.ndarray, eps: float = 1e-5) -> np.ndarray:
    """RMSNorm with unit gain over the last axis: x / sqrt(mean(x^2) + eps)."""
    x = np.asarray(x, dtype=np.float64)
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)


def rope(x: np.ndarray, pos: np.ndarray, theta: float = 10000.0) -> np.ndarray:
    """Rotary position embedding, rotate-half form.

    x: [rows][H][Dh]; pos: [rows].  Dimension i < Dh/2 is paired with i + Dh/2 and
    the pair is rotated by the angle pos * theta**(-2i/Dh)."""
    rows, H, Dh = x.shape
    half = Dh // 2
    inv_freq = theta ** (-2.0 * np.arange(half, dtype=np.float64) / Dh)
    ang = np.asarray(pos, dtype=np.float64)[:, None] * inv_freq[None, :]      # [rows][half]
    c = np.cos(ang)[:, None, :]
    s = np.sin(ang)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def masked_logits(row: np.ndarray, lo: int, hi: int) -> np.ndarray:
    """Logits with every id outside the allowed range [lo, hi) set to -inf."""
    out = np.full_like(row, -np.inf, dtype=np.float64)
    out[lo:hi] = row[lo:hi]
    return out


# ----------------------------------------------------------------------------- Philox
# Philox4x32-10 counter-based generator (Salmon, Moraes, Dror, Shaw, "Parallel random
# numbers: as easy as 1, 2, 3", SC'11): ten rounds of two 32x32->64 multiplies with a
# Weyl-sequence key schedule.
PHILOX_M0 = 0xD2511F53
PHILOX_M1 = 0xCD9E8D57
PHILOX_W0 = 0x9E3779B9
PHILOX_W1 = 0xBB67AE85


def philox4x32_10(ctr, key):
    c0, c1, c2, c3 = (int(v) & MASK32 for v in ctr)
    k0, k1 = (int(v) & MASK32 for v in key)
    for _ in range(10):
        p0 = PHILOX_M0 * c0
        p1 = PHILOX_M1 * c2
        c0, c1, c2, c3 = ((p1 >> 32) ^ c1 ^ k0, p1 & MASK32, (p0 >> 32) ^ c3 ^ k1, p0 & MASK32)
        k0 = (k0 + PHILOX_W0) & MASK32
        k1 = (k1 + PHILOX_W1) & MASK32
    return c0, c1, c2, c3


def uniform_u64(seed: int, step: int, node: int, trial: int) -> int:
    """64 random bits for one acceptance draw: key = seed, counter = (step, node, trial, 0)."""
    x = philox4x32_10((step, node, trial, 0), (seed & MASK32, (seed >> 32) & MASK32))
    return (x[1] << 32) | x[0]


def uniform_u64_tagged(seed: int, step: int, node: int, index: int, tag: int) -> int:
    """64 random bits at key = seed, counter = (step, node, index, tag); tag 0 is the
    acceptance draw above, tag 2 a drafted child (stochastic children)."""
    x = philox4x32_10((step, node, index, tag), (seed & MASK32, (seed >> 32) & MASK32))
    return (x[1] << 32) | x[0]


def draw_below(u64: int, w_total: int) -> int:
    """Uniform integer in [0, w_total): the high 64 bits of the 128-bit product u64 * w_total."""
    return (int(u64) * int(w_total)) >> 64
