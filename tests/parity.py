"""Comparison of GPU results with the oracle's, with near-tie flags.

Token choices are compared exactly.  A choice the two sides may legitimately
make differently -- because fp32 arithmetic on the GPU and fp64 arithmetic in
the oracle put a decision point on opposite sides of a threshold -- is
"flagged" instead of failed; each flag rule bounds how far the GPU's value
can be from the oracle's:

* argmax at T = 0: the top-2 margin of the oracle's logits is below 2 delta,
  delta = max |logit_gpu - logit_oracle| on that row (mapped rows).
* inverse-CDF draw at T > 0: the draw point u*S lies within
  8 (delta/T) sqrt(sum_{i<=j} w_i^2) + 1e-9 S of a breakpoint C_{j-1} or C_j
  (w = oracle weights): the drafter's logit errors shift the cumulative sums
  by about (delta/T) sqrt(sum w^2) when the errors are independent.
* acceptance u_k < r_k: |u_k - r_k| < 1e-5 + 4 (delta/T_d) r_k (delta = 0 when
  both sides read the same drafter logits; T_d the drafter's temperature, no
  drafter term when T_d = 0: q is then one-hot and r_k = p_k(d_k)).
* residual / bonus draw: the draw point is within 8 (delta/T_d) sqrt(sum q^2) +
  1e-8 of a breakpoint (absolute probability units).
"""
from __future__ import annotations

import numpy as np

from oracle import sampling


def argmax_flag(logits: np.ndarray, delta: float) -> bool:
    l = np.asarray(logits, dtype=np.float64)
    l = l[np.isfinite(l)]
    if l.size < 2:
        return False
    top2 = np.partition(l, -2)[-2:]
    return float(top2[1] - top2[0]) < 2.0 * delta + 1e-12


def cdf_margin(w: np.ndarray, u: float):
    """(index chosen, margin to the nearest breakpoint, running sums)."""
    w = np.asarray(w, dtype=np.float64)
    run = np.cumsum(w)
    tot = run[-1]
    tgt = float(u) * tot
    i = sampling.pick_weights(w, u)
    lo = run[i - 1] if i > 0 else 0.0
    return i, min(tgt - lo, run[i] - tgt), run


def draw_flag(logits: np.ndarray, T: float, u: float, delta: float) -> bool:
    """Flag for the drafter's inverse-CDF draw (relative to the total S)."""
    if T == 0.0:
        return argmax_flag(logits, delta)
    w = sampling.softmax_weights(logits, T)
    i, margin, run = cdf_margin(w, u)
    S = run[-1]
    err = 8.0 * (delta / T) * np.sqrt(np.sum(w[: i + 1] ** 2)) + 1e-9 * S
    return margin < err


def accept_flag(u: float, r: float, delta: float, T: float) -> bool:
    extra = 4.0 * (delta / T) * r if T > 0 else 0.0
    return abs(float(u) - float(r)) < 1e-5 + extra


def residual_flag(w: np.ndarray, q: np.ndarray, u: float, delta: float, T: float) -> bool:
    if w.sum() <= 0:
        return True
    i, margin, _ = cdf_margin(w, u)
    err = 1e-8 + (8.0 * (delta / T) * np.sqrt(np.sum(np.asarray(q[: i + 1]) ** 2)) if T > 0 else 0.0)
    return margin < err


def verify_flags(res, target_logits, draft_logits, d2t, drafts, T, u_acc, u_bonus, delta=0.0,
                 T_draft=None):
    """True if any decision of this verification is within its flag window
    (T the target's temperature, T_draft the drafter's; None: T)."""
    from oracle.verify import drafter_probs_on_target
    K = len(drafts)
    Td = T if T_draft is None else float(T_draft)
    if T == 0.0:
        # the oracle's decisions are exact comparisons of identical fp32 inputs
        return False
    for k in range(min(res.accept_len + 1, K)):
        if accept_flag(u_acc[k], res.ratios[k], delta, Td):
            return True
    a = res.accept_len
    tl = np.asarray(target_logits, dtype=np.float64)
    p = sampling.probs(tl[a], T)
    if a < K:
        q = drafter_probs_on_target(draft_logits[a], d2t, tl.shape[1], Td)
        w = np.maximum(p - q, 0.0)
        if w.sum() <= 0:
            w = p
        return residual_flag(w, q, u_bonus, delta, Td)
    return residual_flag(p, np.zeros_like(p), u_bonus, 0.0, T)


def tree_flags(res, target_logits, tokens, parents, T, u_acc, u_bonus) -> bool:
    """True if a decision of this tree verification is within its flag window: a
    tried child's uniform within 1e-5 of its renormalised probability p'(t), or the
    bonus draw point within 1e-6 of the total of a breakpoint (the GPU's target
    probabilities come from fp32 exponentials and chunk sums).  At T = 0 both sides
    compare the same fp32 logits: no flags."""
    from oracle.tree import children_of
    if T == 0.0:
        return False
    tl = np.asarray(target_logits, dtype=np.float64)
    cur = -1
    path = list(res.path) + [None]
    for nxt in path:
        p = sampling.probs(tl[cur + 1], T)
        removed = []
        for c in children_of(parents, cur):
            t = int(tokens[c])
            if t in removed:
                continue
            left = 1.0 - sum(p[r] for r in removed)
            if left > 0.0 and abs(float(u_acc[c]) - p[t] / left) < 1e-5:
                return True
            if nxt is not None and c == nxt:
                break
            removed.append(t)
        if nxt is None:
            w = p.copy()
            w[np.asarray(removed, dtype=np.int64)] = 0.0
            if w.sum() <= 0:
                return True
            _, margin, run = cdf_margin(w, u_bonus)
            return margin < 1e-6 * run[-1] + 1e-12
        cur = int(nxt)
    return False


def tree_near_tie_keys(tree, tol: float) -> set:
    """Path keys of the candidates a near tie may move, over every selection the oracle's
    tree growth made: where two neighbouring values that decide the outcome (the cut
    between kept and dropped, and for a node's top-k children also their rank order)
    are closer than `tol`, every candidate whose value lies within `tol` of that pair."""
    out = set()
    for vals, keys, k, kind in tree.selections:
        pairs = range(min(k, len(vals) - 1)) if kind == "topk" else [k - 1]
        for i in pairs:
            if i + 1 >= len(vals) or not np.isfinite(vals[i + 1]):
                continue
            if vals[i] - vals[i + 1] < tol:
                lo, hi = vals[i + 1] - tol, vals[i] + tol
                out.update(key for v, key in zip(vals, keys) if lo <= v <= hi)
    return out


def tree_mismatch_excused(gpu_keys, oracle_keys, near: set) -> bool:
    """True when every node on which the two trees differ depends on a near tie: the
    node's own path key, or the key of one of its ancestors, is in `near`.  With equal
    node sets the differing positions are compared (a near tie in a rank order changes
    the generation order), otherwise the nodes only one tree holds."""
    g, o = list(gpu_keys), list(oracle_keys)
    if set(g) == set(o):
        diff = {a for a, b in zip(g, o) if a != b} | {b for a, b in zip(g, o) if a != b}
    else:
        diff = set(g) ^ set(o)
    return all(any(key[:j] in near for j in range(1, len(key) + 1)) for key in diff)
