"""Lossless verification of a draft tree (test infrastructure: only tests,
the smoke check and the benchmark's CPU baseline call this module).

The paper serves its drafter through speculative decoding with a top-k
parameter (Section 4, inference settings: top-k 1, i.e. chains); with top-k
> 1 every node of the draft carries the drafter's k most likely tokens as
children, and the target scores all of them in one pass (dynamic draft trees,
discussed among the related drafters).  The children of a node are not
samples from a distribution but deterministic candidates, so the lossless
rule is the target-only one of greedy drafting (the drafter distribution is
one-hot at each candidate), applied to the candidates in turn:

  at node n with target distribution p, for children c_1, c_2, ... in order:
    accept c_i iff u_{c_i} < p'(t_{c_i}), where p' is p with the tokens of the
    children already rejected at n removed and renormalised;
    on acceptance continue from c_i (its own target row), else remove t_{c_i}.
  When no child is accepted, the next token is drawn from p' by inverse CDF
  with u_bonus.

Each step samples exactly from p: accepting c_1 with probability p(t_1), else
drawing from p without t_1, is the same as drawing from p, and so on for the
later candidates.  At T = 0 p is one-hot at the lowest argmax: the walk
follows the child whose token is the target's argmax, and the bonus is that
argmax.  With one child per node this is the chain rule with greedy drafts.

Tree layout: nodes 0..N-1 in topological order (a parent before its
children), parents[i] = -1 for children of the root, else the parent's index;
children are tried in index order.  target_logits row 0 is the root (the
position after the committed prefix), row i + 1 node i.  Node i's uniform is
u_accept[i], used when node i is tried.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from . import sampling


@dataclass
class TreeResult:
    accept_len: int           # accepted nodes on the path
    path: np.ndarray          # [accept_len] node indices, root's child first
    tokens: np.ndarray        # [accept_len + 1]: the path's tokens, then the bonus
    removed: np.ndarray       # tokens rejected at the last node (removed from p)
    last: int                 # node the bonus is drawn at (-1: the root)


def children_of(parents: np.ndarray, n: int) -> np.ndarray:
    """Children of node n (-1: the root) in index order."""
    return np.flatnonzero(np.asarray(parents) == n)


def verify_tree(target_logits: np.ndarray, tokens: np.ndarray, parents: np.ndarray, T: float,
                u_accept: np.ndarray, u_bonus: float) -> TreeResult:
    tl = np.asarray(target_logits, dtype=np.float64)
    tokens = np.asarray(tokens, dtype=np.int64)
    parents = np.asarray(parents, dtype=np.int64)
    cur = -1
    path = []
    while True:
        row = tl[cur + 1]
        kids = children_of(parents, cur)
        removed = []
        nxt = -1
        if T == 0.0:
            star = sampling.argmax_lowest(row)
            for c in kids:
                if tokens[c] == star:
                    nxt = int(c)
                    break
        else:
            p = sampling.probs(row, T)
            for c in kids:
                t = int(tokens[c])
                if t in removed:
                    continue                  # p'(t) = 0: never accepted
                left = 1.0 - sum(p[r] for r in removed)
                if left > 0.0 and float(u_accept[c]) < p[t] / left:
                    nxt = int(c)
                    break
                removed.append(t)
        if nxt < 0:
            break
        path.append(nxt)
        cur = nxt
    row = tl[cur + 1]
    if T == 0.0:
        bonus = sampling.argmax_lowest(row)
    else:
        w = sampling.probs(row, T)
        w[np.asarray(removed, dtype=np.int64)] = 0.0
        if np.sum(w) <= 0.0:                  # every token with mass was a rejected child
            w = sampling.probs(row, T)
        bonus = sampling.pick_weights(w, float(u_bonus))
    out = np.array([tokens[i] for i in path] + [bonus], dtype=np.int64)
    return TreeResult(len(path), np.array(path, dtype=np.int64), out,
                      np.array(removed, dtype=np.int64), cur)


# ---------------------------------------------------------------------------------------
# Drafting a tree (dynamic draft trees with top-k children; the paper's serving setup
# uses top-k 1, i.e. chains)
# ---------------------------------------------------------------------------------------
@dataclass
class DraftTree:
    tokens: np.ndarray        # [N] target ids, topological order (generation order)
    parents: np.ndarray       # [N] -1: child of the root
    scores: np.ndarray        # [N] cumulative log-probability of the node's path
    depths: np.ndarray        # [N] 1 for the root's children
    cand_scores: np.ndarray   # scores of every candidate, in generation order
    min_gap: float = np.inf   # smallest margin of any selection (top-k logits, frontier,
                              # final): where a computation in another precision may differ
    # every selection the growth made, for locating near ties: (values of its best
    # candidates in descending order, their path keys (tuples of target ids from the
    # root), how many it kept, whether the order of the kept ones matters ("topk":
    # children are generated in rank order) or only the cut ("cut"))
    selections: list = None


def top_rows(logits: np.ndarray, k: int) -> np.ndarray:
    """The k drafter rows with the largest logits, best first, ties to the lower row;
    masked rows (-inf) only when fewer than k rows are finite."""
    l = np.asarray(logits, dtype=np.float64)
    order = np.lexsort((np.arange(l.size), -l))      # by logit descending, then row
    return order[:k]


def log_probs(logits: np.ndarray) -> np.ndarray:
    """log softmax at temperature 1 (the drafter's confidence); -inf rows stay -inf."""
    l = np.asarray(logits, dtype=np.float64)
    m = np.max(l)
    return l - m - np.log(np.sum(np.exp(l - m)))


def draft_tree(drafter, seq, tokens, taps, topk: int, depth: int, n_nodes: int) -> DraftTree:
    """Ingest the committed tokens, then grow the tree.

    The root is the last committed row; its k most likely rows (scores log p at
    temperature 1) are the depth-1 candidates.  For depth d = 2 .. `depth` every
    node of the frontier (the k best candidates of the previous depth; depth 1: all
    of them) runs through the drafter at position committed + (its depth - 1), with
    its parent's hidden state as the conditioning input, attending to the committed
    context and to its own ancestors (each branch has its own copy of the cache
    beyond the context); its k most likely rows become candidates with the parent's
    score plus their log probability.  Finally the n_nodes best candidates (score,
    then generation order) form the tree, listed in generation order."""
    import copy
    gaps = []
    selections = []

    def gap(values, k):           # margin between the k-th and (k+1)-th largest values
        v = np.sort(np.asarray(values, dtype=np.float64)[np.isfinite(values)])[::-1]
        if len(v) > k:
            gaps.append(v[k - 1] - v[k])

    def record(values, keys, k, kind, extra=16):
        values = np.asarray(values, dtype=np.float64)
        order = np.lexsort((np.arange(values.size), -values))[: k + extra]
        selections.append((values[order], [keys(int(i)) for i in order], k, kind))

    def key_of(i):                # path key of candidate i: target ids from the root
        out = []
        while i >= 0:
            out.append(cands[i][0])
            i = cands[i][1]
        return tuple(out[::-1])

    g_root = drafter.ingest(seq, tokens, taps)
    L = seq.length
    cands = []      # (token, parent candidate index, score, depth)
    lp = log_probs(drafter.logits(g_root))
    gap(drafter.logits(g_root), topk)
    record(drafter.logits(g_root), lambda r: (int(drafter.d2t[r]),), topk, "topk")
    for r in top_rows(drafter.logits(g_root), topk):
        cands.append((int(drafter.d2t[r]), -1, float(lp[r]), 1))
    state = {}      # candidate index -> (branch cache, hidden state g)
    frontier = list(range(len(cands)))
    for d in range(2, depth + 1):
        new = []
        for f in frontier:
            tok, par, sc, dep = cands[f]
            base, g_par = (seq, g_root) if par < 0 else state[par]
            br = copy.deepcopy(base)
            g = drafter.forward_row(br, tok, g_par, L + dep - 1)
            state[f] = (br, g)
            l = drafter.logits(g)
            lpf = log_probs(l)
            gap(l, topk)
            record(l, lambda r, f=f: key_of(f) + (int(drafter.d2t[r]),), topk, "topk")
            for r in top_rows(l, topk):
                new.append(len(cands))
                cands.append((int(drafter.d2t[r]), f, sc + float(lpf[r]), dep + 1))
        order = sorted(new, key=lambda i: (-cands[i][2], i))
        if d < depth:
            gap([cands[i][2] for i in new], topk)
            record([cands[i][2] for i in new], lambda j, new=new: key_of(new[j]), topk, "cut")
        frontier = sorted(order[:topk])
    allsc = np.array([c[2] for c in cands])
    gap(allsc, n_nodes)
    record(allsc, key_of, n_nodes, "cut")
    pick = sorted(sorted(range(len(cands)), key=lambda i: (-cands[i][2], i))[:n_nodes])
    index = {c: j for j, c in enumerate(pick)}
    toks = np.array([cands[i][0] for i in pick], dtype=np.int64)
    pars = np.array([index[cands[i][1]] if cands[i][1] >= 0 else -1 for i in pick], dtype=np.int64)
    return DraftTree(toks, pars, np.array([cands[i][2] for i in pick]),
                     np.array([cands[i][3] for i in pick], dtype=np.int64), allsc,
                     min(gaps) if gaps else np.inf, selections)
