"""Pins of the oracle's draft-tree verification against the mathematics.

* A tree with one child per node is a chain of greedy drafts: the result
  equals the chain rule with q one-hot (an independently pinned function).
* Losslessness: the first committed token is distributed as p_root and, given
  that a child was accepted, the next one as that child's p (chi-square), for
  a tree whose root has several children (including a duplicate token and a
  token the target gives no mass); a planted mistake (accepting a later child
  with p(t) instead of the renormalised p'(t)) is rejected.
* Closed forms: the probability that child i of the root is accepted is
  p(t_i) (each step of the walk samples from p); the bonus after rejecting
  every child is distributed as p without the children's tokens.
* Greedy (T = 0): the accepted path is the longest path whose every token is
  the argmax of its parent's row (brute force over random trees), and the
  bonus is the argmax at the path's end.
"""
import numpy as np
import pytest
from scipy import stats

from oracle import sampling
from oracle.tree import children_of, verify_tree
from oracle.verify import verify


def _random_tree(rng, n, width):
    """Random topological tree: node i's parent is -1 or an earlier node."""
    parents = np.empty(n, dtype=np.int64)
    for i in range(n):
        parents[i] = -1 if i < width or rng.random() < 0.2 else int(rng.integers(0, i))
    return parents


def test_single_child_tree_is_the_greedy_draft_chain():
    rng = np.random.default_rng(11)
    V, K = 7, 5
    for trial in range(300):
        tl = rng.standard_normal((K + 1, V)) * 1.5
        drafts = rng.integers(0, V, size=K)
        dl = rng.standard_normal((K, V))
        dl[np.arange(K), drafts] = 10.0           # the chain's drafts are the drafter's argmax
        u = rng.random(K)
        ub = float(rng.random())
        T = float(rng.choice([0.0, 0.7, 1.0]))
        parents = np.arange(-1, K - 1)
        tr = verify_tree(tl, drafts, parents, T, u, ub)
        ch = verify(tl, dl, np.arange(V), drafts, T, u, ub, T_draft=0.0)
        assert tr.accept_len == ch.accept_len
        assert list(tr.tokens) == list(ch.tokens[: ch.accept_len + 1])


def _first_tokens(p_rows, tokens, parents, T, n, seed, mistake=False):
    rng = np.random.default_rng(seed)
    first, second = [], []
    for _ in range(n):
        u = rng.random(len(tokens))
        ub = float(rng.random())
        if mistake:
            r = _verify_without_renormalising(p_rows, tokens, parents, u, ub)
        else:
            r = verify_tree(np.log(p_rows) * T, tokens, parents, T, u, ub)
        first.append(int(r.tokens[0]))
        second.append((int(r.path[0]) if r.accept_len else -1, int(r.tokens[1]) if len(r.tokens) > 1 else -1))
    return np.array(first), second


def _verify_without_renormalising(p_rows, tokens, parents, u, ub):
    """The planted mistake: child i accepted with p(t_i), not p(t_i) / (1 - rejected)."""
    cur, path, removed = -1, [], []
    while True:
        p = p_rows[cur + 1]
        nxt = -1
        for c in children_of(parents, cur):
            if u[c] < p[tokens[c]]:
                nxt = int(c)
                break
            removed.append(int(tokens[c]))
        if nxt < 0:
            break
        path.append(nxt)
        cur = nxt
    w = p_rows[cur + 1].copy()
    w[removed] = 0.0
    bonus = sampling.pick_weights(w, ub)

    class R:
        pass
    r = R()
    r.accept_len, r.path = len(path), np.array(path)
    r.tokens = np.array([tokens[i] for i in path] + [bonus])
    return r


def _tree_case():
    V = 6
    rng = np.random.default_rng(5)
    # root children: tokens 2, 0, 2 (duplicate), 5 (no target mass); node 0 has two children
    tokens = np.array([2, 0, 2, 5, 1, 3])
    parents = np.array([-1, -1, -1, -1, 0, 0])
    p_rows = rng.dirichlet(np.ones(V), size=len(tokens) + 1)
    p_rows[0, 5] = 0.0
    p_rows[0] /= p_rows[0].sum()
    return V, tokens, parents, np.maximum(p_rows, 1e-300)


@pytest.mark.parametrize("seed", [0, 1])
def test_tree_verification_is_lossless(seed):
    V, tokens, parents, p_rows = _tree_case()
    n = 30000
    first, second = _first_tokens(p_rows, tokens, parents, 1.0, n, seed)
    counts = np.bincount(first, minlength=V)
    exp = p_rows[0] * n
    keep = exp > 1e-9
    assert counts[~keep].sum() == 0
    assert stats.chisquare(counts[keep], exp[keep]).pvalue > 1e-4
    # given node 0 (token 2) accepted, the next token follows p of node 0's row
    nxt = np.array([t for (node, t) in second if node == 0])
    c2 = np.bincount(nxt, minlength=V)
    assert stats.chisquare(c2, p_rows[1] * len(nxt)).pvalue > 1e-4


def test_tree_verification_rejects_a_planted_mistake():
    V, tokens, parents, p_rows = _tree_case()
    n = 30000
    first, _ = _first_tokens(p_rows, tokens, parents, 1.0, n, 3, mistake=True)
    counts = np.bincount(first, minlength=V)
    exp = p_rows[0] * n
    keep = exp > 1e-9
    assert stats.chisquare(counts[keep], exp[keep]).pvalue < 1e-6


def test_tree_closed_forms():
    V, tokens, parents, p_rows = _tree_case()
    rng = np.random.default_rng(9)
    n = 40000
    acc = np.zeros(len(tokens))
    bon = np.zeros(V)
    nbon = 0
    for _ in range(n):
        u = rng.random(len(tokens))
        ub = float(rng.random())
        r = verify_tree(np.log(p_rows), tokens, parents, 1.0, u, ub)
        if r.accept_len:
            acc[r.path[0]] += 1
        else:
            bon[r.tokens[0]] += 1
            nbon += 1
    p = p_rows[0]
    # child i of the root is accepted with probability p(t_i); the duplicate never
    assert abs(acc[0] / n - p[2]) < 4 * np.sqrt(p[2] / n)
    assert abs(acc[1] / n - p[0]) < 4 * np.sqrt(p[0] / n)
    assert acc[2] == 0 and acc[3] == 0
    # after rejecting every child: p without the children's tokens
    w = p.copy()
    w[[2, 0, 5]] = 0.0
    w /= w.sum()
    assert bon[[0, 2, 5]].sum() == 0
    keep = w > 1e-12
    assert stats.chisquare(bon[keep], w[keep] * nbon).pvalue > 1e-4


def _greedy_path(tl, tokens, parents):
    cur, path = -1, []
    while True:
        star = int(np.argmax(tl[cur + 1]))
        nxt = [int(c) for c in range(len(tokens)) if parents[c] == cur and tokens[c] == star]
        if not nxt:
            return path, star
        cur = nxt[0]
        path.append(cur)


def test_greedy_tree_follows_argmax_children():
    rng = np.random.default_rng(21)
    V = 5
    for trial in range(500):
        n = int(rng.integers(0, 12))
        parents = _random_tree(rng, n, int(rng.integers(1, 4)))
        tokens = rng.integers(0, V, size=n)
        tl = rng.standard_normal((n + 1, V))
        r = verify_tree(tl, tokens, parents, 0.0, rng.random(n), 0.5)
        path, star = _greedy_path(tl, tokens, parents)
        assert list(r.path) == path
        assert int(r.tokens[-1]) == star
        for a, b in zip(path[1:], path[:-1]):
            assert parents[a] == b


def test_empty_tree_samples_the_root():
    rng = np.random.default_rng(2)
    tl = rng.standard_normal((1, 8))
    for u in (0.0, 0.3, 0.9):
        r = verify_tree(tl, np.zeros(0, np.int64), np.zeros(0, np.int64), 1.0, np.zeros(0), u)
        assert r.accept_len == 0
        assert int(r.tokens[0]) == sampling.pick(tl[0], 1.0, u)


# ----------------------------------------------------------------------------------------
# tree drafting
# ----------------------------------------------------------------------------------------
def _tiny_drafter(dtype="bf16"):
    import synth
    from oracle.drafter import Drafter, Sequence
    w = synth.Workload(name="tree_pin", cfg_id=131, dtype=dtype, n_layers=2, d_model=64,
                       n_q_heads=4, n_kv_heads=2, head_dim=16, d_ffn=96, vocab_draft=61,
                       vocab_target=61, target_hidden=24, batch=1, K=3, prefill="ingest",
                       gains="normal")
    dr = Drafter(w, synth.make_weights(w), synth.make_d2t(w))
    rng = np.random.default_rng(4)
    toks = rng.integers(0, w.vocab_target, 9)
    taps = rng.standard_normal((9, 3 * w.target_hidden))
    return w, dr, Sequence, toks, taps


def test_tree_with_one_child_per_node_is_the_greedy_chain():
    from oracle.tree import draft_tree
    w, dr, Sequence, toks, taps = _tiny_drafter()
    for K in (1, 3, 5):
        s1, s2 = Sequence(w, 64), Sequence(w, 64)
        t = draft_tree(dr, s1, toks, taps, 1, K, K)
        drafts, _, _, _ = dr.draft(s2, toks, taps, K, 0.0, np.zeros(K))
        assert list(t.tokens) == list(drafts)
        assert list(t.parents) == list(range(-1, K - 1))


def test_tree_nodes_match_independent_path_replays():
    """Every selected node's score is the sum of log-probabilities along its path,
    recomputed by replaying the path through a fresh copy of the committed cache,
    and its children are among the top-k rows of the replayed logits; the
    selection is the n best candidates and contains every selected node's parent."""
    import copy
    from oracle.tree import draft_tree, log_probs, top_rows
    w, dr, Sequence, toks, taps = _tiny_drafter()
    topk, depth, n = 3, 4, 12
    seq = Sequence(w, 64)
    t = draft_tree(dr, seq, toks, taps, topk, depth, n)
    base = Sequence(w, 64)
    g0 = dr.ingest(base, toks, taps)
    L = base.length
    inv = {int(dr.d2t[r]): r for r in range(w.vocab_draft) if dr.d2t[r] >= 0}
    for i in range(n):
        path = [i]
        while t.parents[path[-1]] >= 0:
            path.append(int(t.parents[path[-1]]))
        path = path[::-1]
        br = copy.deepcopy(base)
        g, score = g0, 0.0
        for j, node in enumerate(path):
            l = dr.logits(g)
            r = inv[int(t.tokens[node])]
            assert r in top_rows(l, topk)
            score += log_probs(l)[r]
            if j + 1 < len(path):
                g = dr.forward_row(br, int(t.tokens[node]), g, L + j)
        assert abs(score - t.scores[i]) < 1e-9
        assert t.depths[i] == len(path)
    best = np.sort(t.cand_scores)[::-1][:n]
    assert np.allclose(np.sort(t.scores)[::-1], best)
    assert all(p < i for i, p in enumerate(t.parents))


def test_tree_is_independent_of_taps_with_zero_expansion():
    """Eq. 3: with the c-slot columns zero the tree does not depend on the taps."""
    import synth
    from oracle.drafter import Drafter, Sequence
    from oracle.tree import draft_tree
    w = synth.Workload(name="tree_zero", cfg_id=132, dtype="bf16", n_layers=1, d_model=64,
                       n_q_heads=2, n_kv_heads=1, head_dim=32, d_ffn=64, vocab_draft=53,
                       vocab_target=53, target_hidden=16, batch=1, K=3, prefill="ingest",
                       expansion="zero")
    dr = Drafter(w, synth.make_weights(w), synth.make_d2t(w))
    rng = np.random.default_rng(8)
    toks = rng.integers(0, w.vocab_target, 6)
    a = draft_tree(dr, Sequence(w, 32), toks, rng.standard_normal((6, 48)), 3, 3, 8)
    b = draft_tree(dr, Sequence(w, 32), toks, rng.standard_normal((6, 48)) * 5, 3, 3, 8)
    assert list(a.tokens) == list(b.tokens) and list(a.parents) == list(b.parents)
    assert np.array_equal(a.scores, b.scores)
