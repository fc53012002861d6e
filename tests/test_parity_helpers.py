"""The near-tie localisation the GPU tree-growth comparison uses (tests/parity.py):
a mismatch is excused only by a near tie on the mismatching node's own path."""
import numpy as np

from . import parity


def _tree():
    import synth
    from oracle.drafter import Drafter, Sequence
    from oracle.tree import draft_tree
    w = synth.Workload(name="tree_loc", cfg_id=133, dtype="bf16", n_layers=1, d_model=64,
                       n_q_heads=2, n_kv_heads=1, head_dim=32, d_ffn=64, vocab_draft=53,
                       vocab_target=53, target_hidden=16, batch=1, K=3, prefill="ingest")
    dr = Drafter(w, synth.make_weights(w), synth.make_d2t(w))
    rng = np.random.default_rng(9)
    toks = rng.integers(0, w.vocab_target, 6)
    return draft_tree(dr, Sequence(w, 32), toks, rng.standard_normal((6, 48)), 3, 3, 9)


def _keys(tokens, parents):
    out = []
    for i in range(len(tokens)):
        k, j = [], i
        while j >= 0:
            k.append(int(tokens[j]))
            j = int(parents[j])
        out.append(tuple(k[::-1]))
    return out


def test_near_tie_localisation():
    t = _tree()
    ok = _keys(t.tokens, t.parents)
    # every selection is recorded with its candidates' path keys
    assert len(t.selections) >= 1 + 3 + 1
    assert all(len(v) == len(k) for v, k, _, _ in t.selections)
    # the last node's token replaced: a difference no near tie explains ...
    tk = t.tokens.copy()
    tk[-1] = (int(tk[-1]) + 1) % 53
    gk = _keys(tk, t.parents)
    assert not parity.tree_mismatch_excused(gk, ok, set())
    # ... nor one on another branch ...
    other = next(k for k in ok if k[0] != ok[-1][0])
    assert not parity.tree_mismatch_excused(gk, ok, {other})
    # ... but one on its path does, and so does a near tie between the two candidates
    # themselves (a tie names both), not a tie naming only one of them
    assert parity.tree_mismatch_excused(gk, ok, {ok[-1][:1]})
    assert parity.tree_mismatch_excused(gk, ok, {ok[-1], gk[-1]})
    assert not parity.tree_mismatch_excused(gk, ok, {ok[-1]})
    # no tie is that close; every selection is, at an absurd tolerance
    assert parity.tree_near_tie_keys(t, 1e-12) == set()
    assert parity.tree_mismatch_excused(gk, ok, parity.tree_near_tie_keys(t, 1e9))
    # identical trees need no excuse
    assert parity.tree_mismatch_excused(ok, ok, set())
