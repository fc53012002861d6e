"""Turning a distribution and a uniform into one token.

The paper does not state how a token is drawn from a distribution given a
uniform.  The rule used throughout (drafter sampling, residual resampling,
bonus sampling) is the inverse CDF over token ids in ascending order: the
chosen id is the smallest i whose running sum of weights exceeds u times the
total.  At temperature 0 the choice is the argmax, ties to the lowest id.
"""
from __future__ import annotations

import numpy as np


def argmax_lowest(x: np.ndarray) -> int:
    """Index of the maximum, lowest index on ties (numpy's argmax does this)."""
    return int(np.argmax(x))


def pick_weights(w: np.ndarray, u: float) -> int:
    """Inverse CDF over non-negative weights w (ascending ids): smallest i with
    w_0 + ... + w_i > u * sum(w).  Callers guarantee sum(w) > 0."""
    w = np.asarray(w, dtype=np.float64)
    run = np.cumsum(w)                 # running sums in ascending id order
    target = float(u) * run[-1]
    above = run > target
    if above.any():
        return int(np.argmax(above))   # first id whose running sum exceeds the target
    return int(np.flatnonzero(w > 0.0)[-1])   # only through rounding as u -> 1


def softmax_weights(logits: np.ndarray, T: float) -> np.ndarray:
    """exp((l - max) / T); -inf logits get weight 0."""
    l = np.asarray(logits, dtype=np.float64)
    m = np.max(l)
    return np.exp((l - m) / T)


def pick(logits: np.ndarray, T: float, u: float) -> int:
    """Token index from logits at temperature T (T = 0: argmax)."""
    if T == 0.0:
        return argmax_lowest(np.asarray(logits, dtype=np.float64))
    return pick_weights(softmax_weights(logits, T), u)


def probs(logits: np.ndarray, T: float) -> np.ndarray:
    """softmax(l / T); at T = 0 the one-hot of the lowest argmax."""
    l = np.asarray(logits, dtype=np.float64)
    if T == 0.0:
        p = np.zeros_like(l)
        p[argmax_lowest(l)] = 1.0
        return p
    w = softmax_weights(l, T)
    return w / np.sum(w)
