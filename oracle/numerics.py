"""Elementwise building blocks of the drafter, in float64.

These are the standard definitions of the pieces the drafter inherits from its
source LM unchanged (Section 3.3 keeps the feed-forward blocks, the norms and the
other pretrained parts of the source model as they are); the paper names the
source (Qwen3-4B, Section 4) but not the formulas, so each is the Qwen3
definition.
"""
from __future__ import annotations

import numpy as np


def rmsnorm(x: np.ndarray, gain: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * gain over the last axis."""
    x = np.asarray(x, dtype=np.float64)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * np.asarray(gain, dtype=np.float64)


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def rope_rotate_half(x: np.ndarray, pos: int, theta: float) -> np.ndarray:
    """Rotary position embedding, rotate-half convention.

    x: [..., hd].  Pair i (i < hd/2) is (x_i, x_{i+hd/2}), rotated by the angle
    pos * theta^(-2i/hd)."""
    x = np.asarray(x, dtype=np.float64)
    hd = x.shape[-1]
    half = hd // 2
    inv_freq = theta ** (-(2.0 * np.arange(half, dtype=np.float64)) / hd)
    ang = float(pos) * inv_freq
    c, s = np.cos(ang), np.sin(ang)
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray) -> np.ndarray:
    """Grouped-query scaled dot-product attention of one query position.

    q: [n_q, hd]; k, v: [n, n_kv, hd] (every cached position the query may see).
    Query head h reads key/value head floor(h * n_kv / n_q).  Scale 1/sqrt(hd),
    softmax over positions.  Returns [n_q, hd]."""
    n_q, hd = q.shape
    n_kv = k.shape[1]
    out = np.empty((n_q, hd), dtype=np.float64)
    for h in range(n_q):
        g = (h * n_kv) // n_q
        scores = k[:, g, :] @ q[h] / np.sqrt(hd)
        m = np.max(scores)
        p = np.exp(scores - m)
        p /= np.sum(p)
        out[h] = p @ v[:, g, :]
    return out


def bf16_rne(x: np.ndarray) -> np.ndarray:
    """Round each value to the nearest bfloat16 value, ties to even.

    bfloat16 keeps 8 significant bits; values are returned as float64."""
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)                 # x = m * 2^e, 0.5 <= |m| < 1
    return np.ldexp(np.round(m * 256.0), e - 8)
