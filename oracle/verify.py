"""Lossless verification of a chain of drafts (the standard speculative
decoding acceptance rule, which the paper keeps unchanged: Section 3.1, and
the losslessness claim of Section 1).

Index convention: drafts d_0..d_{K-1} were drawn from the drafter's
distributions q_0..q_{K-1}; the target's verify pass gives p_0..p_K, where
p_k is the next-token distribution after the committed prefix followed by
d_0..d_{k-1}.  Draft k is accepted with probability min(1, p_k(d_k)/q_k(d_k))
(decided as u_k < min(1, p/q) with a given uniform); at the first rejection a
replacement is drawn from the normalised residual max(0, p_a - q_a); if every
draft is accepted a bonus token is drawn from p_K.  At temperature 0 both
distributions are one-hot at their argmax, which makes this a greedy prefix
match followed by the target's argmax.

The drafter may draw its drafts at a temperature of its own (T_draft) while the
target is sampled at T.  The rule is unchanged: q is the distribution the
drafts were actually drawn from.  With T_draft = 0 (greedy drafting: the
top-1 chain of the paper's serving setup, Section 4 "Inference settings and
metrics" and the serving configuration of the adaptation appendix) q is
one-hot at the drafter's argmax, so draft k is accepted with probability
p_k(d_k) and a rejected position is redrawn from p_a with d_a removed.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from . import sampling


@dataclass
class VerifyResult:
    accept_len: int
    mask: np.ndarray          # [K] uint8
    tokens: np.ndarray        # [K + 1] int64: d_0..d_{a-1}, replacement/bonus, then -1
    ratios: np.ndarray        # [K] the acceptance thresholds min(1, p/q) (T > 0; else 0/1)
    residual_used: bool       # the replacement came from the residual (not from p)


def drafter_probs_on_target(draft_logits: np.ndarray, d2t: np.ndarray, V_T: int,
                            T: float) -> np.ndarray:
    """q over target ids: the drafter's softmax(l/T) carried through d2t;
    target ids that no drafter row maps to get probability 0."""
    qd = sampling.probs(draft_logits, T)
    q = np.zeros(V_T, dtype=np.float64)
    m = d2t >= 0
    q[d2t[m]] = qd[m]
    return q


def verify(target_logits: np.ndarray, draft_logits: np.ndarray, d2t: np.ndarray,
           drafts: np.ndarray, T: float, u_accept: np.ndarray, u_bonus: float,
           residual_fn=None, T_draft=None) -> VerifyResult:
    """target_logits [K+1, V_T]; draft_logits [K, V_d]; drafts [K] target ids.
    T is the target's temperature, T_draft the drafter's (None: the same as T)."""
    Td = T if T_draft is None else float(T_draft)
    tl = np.asarray(target_logits, dtype=np.float64)
    K = len(drafts)
    V_T = tl.shape[1]
    d2t = np.asarray(d2t, dtype=np.int64)
    residual_fn = residual_fn or (lambda p, q: np.maximum(p - q, 0.0))
    mask = np.zeros(K, dtype=np.uint8)
    ratios = np.zeros(K, dtype=np.float64)
    a = 0
    q_rows = []
    while a < K:
        p = sampling.probs(tl[a], T)
        q = drafter_probs_on_target(draft_logits[a], d2t, V_T, Td)
        q_rows.append(q)
        d = int(drafts[a])
        pd, qd = p[d], q[d]
        if qd > 0.0:
            r = min(1.0, pd / qd)
        else:                    # min(1, p/0): 1 where the target has mass, else 0
            r = 1.0 if pd > 0.0 else 0.0
        ratios[a] = r
        if float(u_accept[a]) < r:
            mask[a] = 1
            a += 1
        else:
            break
    tokens = np.full(K + 1, -1, dtype=np.int64)
    tokens[:a] = np.asarray(drafts[:a], dtype=np.int64)
    residual_used = False
    p_a = sampling.probs(tl[a], T)
    if T == 0.0:
        tokens[a] = sampling.argmax_lowest(tl[a])
    elif a < K:
        w = residual_fn(p_a, q_rows[a])
        if np.sum(w) > 0.0:
            tokens[a] = sampling.pick_weights(w, float(u_bonus))
            residual_used = True
        else:                               # degenerate residual: fall back to p_a
            tokens[a] = sampling.pick_weights(p_a, float(u_bonus))
    else:
        tokens[a] = sampling.pick_weights(p_a, float(u_bonus))
    return VerifyResult(a, mask, tokens, ratios, residual_used)
