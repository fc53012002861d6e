"""Pins of the oracle's block drafting (the EAGLE-style interface of the DFlash
ablation) against what the appendix and the mathematics fix.

* Against an independent decoder: with the same conditioning input at every
  position, the drafter is a Qwen3 model with Q/K/V biases W^c s (pinned for the
  chain); a block's rows must then be that model's logits at the anchor and at the
  mask positions that follow it, causally (positions, the mask token, the shift of
  one between a row and the token it predicts, the broadcast of the anchor's input).
* A block of one proposal is the chain's first draft.
* With zero expansion (Eq. 3) the block does not depend on the taps.
* Verifying independent proposals with the chain rule is lossless: the first two
  committed tokens follow p_0 and p_1 (chi-square) when each draft is drawn from
  its own row q_k; verifying the second draft against the first row's q instead
  (a planted mistake) is rejected.
"""
import numpy as np
from scipy import stats

import synth
from oracle import sampling
from oracle.block import draft_block
from oracle.drafter import Drafter, Sequence
from oracle.verify import verify

from .test_oracle_drafter_pins import _hf_logits, _hf_model, _tiny


def test_block_rows_equal_qwen3_with_qkv_bias_at_the_block_positions():
    w = _tiny(expansion="normal", d_model=64, n_q_heads=8, n_kv_heads=2, head_dim=8)
    weights = synth.make_weights(w)
    dr = Drafter(w, weights, np.arange(w.vocab_draft))
    toks = synth.prompt_tokens(w, 2, 13)
    tap = np.random.default_rng(17).standard_normal(w.tap_width)
    mask, K = 5, 6
    _, logits, _, committed = draft_block(dr, Sequence(w, 40), toks, np.tile(tap, (13, 1)), K, 0.0,
                                          np.zeros(K), mask)
    assert committed == 13
    s = np.asarray(weights["w_c"], dtype=np.float64) @ tap
    full = np.concatenate([toks, np.full(K - 1, mask)])
    ref = _hf_logits(_hf_model(w, weights, bias_s=s), full)[12:12 + K]
    np.testing.assert_allclose(logits, ref, atol=2e-6, rtol=0)
    # the mask rows see each other (the block is not K copies of one row)
    assert np.max(np.abs(logits[1] - logits[2])) > 1e-3


def test_block_of_one_is_the_chain_first_draft():
    w = _tiny()
    weights = synth.make_weights(w)
    dr = Drafter(w, weights, np.arange(w.vocab_draft))
    rng = np.random.default_rng(3)
    toks = rng.integers(0, w.vocab_target, 7)
    taps = rng.standard_normal((7, w.tap_width))
    for T, u in ((0.0, 0.5), (1.0, 0.3), (0.7, 0.9)):
        a = draft_block(dr, Sequence(w, 20), toks, taps, 1, T, [u], 3)
        b = dr.draft(Sequence(w, 20), toks, taps, 1, T, [u])
        assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1]) and a[3] == b[3]


def test_block_is_independent_of_taps_with_zero_expansion():
    w = _tiny(expansion="zero")
    weights = synth.make_weights(w)
    dr = Drafter(w, weights, np.arange(w.vocab_draft))
    rng = np.random.default_rng(4)
    toks = rng.integers(0, w.vocab_target, 9)
    a = draft_block(dr, Sequence(w, 30), toks, rng.standard_normal((9, w.tap_width)), 5, 1.0,
                    np.full(5, 0.4), 7)
    b = draft_block(dr, Sequence(w, 30), toks, rng.standard_normal((9, w.tap_width)) * 9, 5, 1.0,
                    np.full(5, 0.4), 7)
    assert np.array_equal(a[1], b[1]) and np.array_equal(a[0], b[0])


def _committed(p_rows, q_rows, n, seed, verify_q=None):
    """First two committed tokens over n trials; drafts d_k ~ q_k independently."""
    rng = np.random.default_rng(seed)
    V = p_rows.shape[1]
    ql = np.log(q_rows)
    vq = ql if verify_q is None else np.log(verify_q)
    first, second = [], []
    for _ in range(n):
        u = rng.random(2)
        d = np.array([sampling.pick(ql[k], 1.0, float(u[k])) for k in range(2)])
        r = verify(np.log(p_rows), vq, np.arange(V), d, 1.0, rng.random(2), float(rng.random()),
                   T_draft=1.0)
        first.append(int(r.tokens[0]))
        if r.accept_len >= 1:
            second.append(int(r.tokens[1]))
    return np.array(first), np.array(second)


def test_independent_block_proposals_verify_losslessly():
    rng = np.random.default_rng(8)
    V = 6
    p = rng.dirichlet(np.ones(V), size=3)
    q = rng.dirichlet(np.ones(V) * 0.7, size=2)
    for seed in (0, 1):
        f, s2 = _committed(p, q, 30000, seed)
        assert stats.chisquare(np.bincount(f, minlength=V), p[0] * len(f)).pvalue > 1e-4
        assert stats.chisquare(np.bincount(s2, minlength=V), p[1] * len(s2)).pvalue > 1e-4
    # planted mistake: the second draft checked against the first row's distribution
    _, s2 = _committed(p, q, 30000, 2, verify_q=np.stack([q[0], q[0]]))
    assert stats.chisquare(np.bincount(s2, minlength=V), p[1] * len(s2)).pvalue < 1e-6
