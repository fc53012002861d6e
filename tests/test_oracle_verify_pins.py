"""Pins of the oracle's sampling and verification against the mathematics.

The paper keeps the standard acceptance rule (Section 3.1) and relies on its
guarantee that committed tokens follow the target distribution exactly
(Section 1).  These tests check the oracle against that guarantee and its
consequences rather than against itself:

* inverse-CDF sampling equals numpy's searchsorted on the cumulative sum;
* greedy verification accepts exactly the longest prefix of target argmaxes;
* losslessness: over many trials the first committed token is distributed as
  p_0 and, given d_0 was accepted, the second as p_1 (chi-square); the same
  test rejects a planted mistake (resampling from p instead of the residual);
* the acceptance frequency of draft k is sum_v min(p_k, q_k);
* q = p accepts everything; K = 0 is plain sampling from p_0; target ids that
  no drafter row reaches have q = 0 and are still reachable through the
  residual;
* greedy drafting against a sampled target (q one-hot): lossless by
  chi-square, acceptance frequency p_k(d_k), a rejected position redrawn from
  p_k without d_k (closed forms), and a planted mistake (treating greedy drafts
  as sampled at the target's temperature) is rejected.
"""
import numpy as np
import pytest
from scipy import stats

from oracle import sampling
from oracle.verify import drafter_probs_on_target, verify


def test_pick_equals_searchsorted():
    rng = np.random.default_rng(0)
    for trial in range(300):
        n = int(rng.integers(1, 60))
        w = rng.exponential(size=n) * (rng.random(n) < 0.7)
        if w.sum() == 0:
            w[int(rng.integers(n))] = 1.0
        u = float(rng.integers(0, 1 << 24)) * 2.0 ** -24
        ref = int(np.searchsorted(np.cumsum(w), u * np.cumsum(w)[-1], side="right"))
        assert sampling.pick_weights(w, u) == ref


def test_pick_temperature_zero_is_lowest_argmax_and_onehot():
    l = np.array([0.5, 2.0, -1.0, 2.0, 1.0])
    assert sampling.pick(l, 0.0, 0.3) == 1
    onehot = np.full(7, -np.inf)
    onehot[4] = 0.0
    for u in (0.0, 0.5, 1 - 2 ** -24):
        assert sampling.pick(onehot, 1.0, u) == 4


def _rand_logits(rng, n, scale=1.0):
    return rng.standard_normal(n) * scale


def test_greedy_verify_is_longest_argmax_prefix():
    rng = np.random.default_rng(1)
    V, K = 9, 5
    d2t = np.arange(V)
    for trial in range(400):
        tl = _rand_logits(rng, (K + 1, V))
        dl = _rand_logits(rng, (K, V))
        best = np.argmax(tl, axis=1)
        j = int(rng.integers(0, K + 1))       # first mismatch position (K: none)
        drafts = best[:K].copy()
        if j < K:
            drafts[j] = (best[j] + 1 + int(rng.integers(V - 1))) % V
        for i in range(j + 1, K):
            drafts[i] = int(rng.integers(V))
        r = verify(tl, dl, d2t, drafts, 0.0, np.zeros(K), 0.0)
        assert r.accept_len == j
        assert list(r.mask) == [1] * j + [0] * (K - j)
        assert list(r.tokens[:j]) == list(drafts[:j])
        assert r.tokens[j] == best[j]


def _draw_drafts(q_rows, u):
    return np.array([sampling.pick_weights(q, x) for q, x in zip(q_rows, u)])


def _lossless_counts(p_logits, q_logits, T, n, seed, residual_fn=None):
    """Sample drafts from q, verify against p; histogram the first committed
    token and, when d_0 was accepted, the second."""
    rng = np.random.default_rng(seed)
    K, V = q_logits.shape
    d2t = np.arange(V)
    q_rows = [sampling.probs(q_logits[k], T) for k in range(K)]
    first = np.zeros(V, dtype=np.int64)
    second = np.zeros(V, dtype=np.int64)
    for _ in range(n):
        ud = rng.random(K)
        drafts = _draw_drafts(q_rows, ud)
        r = verify(p_logits, q_logits, d2t, drafts, T, rng.random(K), rng.random(),
                   residual_fn=residual_fn)
        first[r.tokens[0]] += 1
        if r.accept_len >= 1:
            second[r.tokens[1]] += 1
    return first, second


def _chi2_p(counts, probs):
    exp = probs * counts.sum()
    keep = exp > 0
    assert counts[~keep].sum() == 0
    return stats.chisquare(counts[keep], exp[keep]).pvalue


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_lossless_first_and_second_token(seed):
    rng = np.random.default_rng(100 + seed)
    V, K, T = 10, 2, 1.0
    p_logits = _rand_logits(rng, (K + 1, V), 1.5)
    q_logits = _rand_logits(rng, (K, V), 1.5)
    first, second = _lossless_counts(p_logits, q_logits, T, 30000, seed)
    assert _chi2_p(first, sampling.probs(p_logits[0], T)) > 1e-4
    assert _chi2_p(second, sampling.probs(p_logits[1], T)) > 1e-4


def test_lossless_test_rejects_planted_residual_mistake():
    rng = np.random.default_rng(7)
    V, K, T = 10, 2, 1.0
    p_logits = _rand_logits(rng, (K + 1, V), 1.5)
    q_logits = _rand_logits(rng, (K, V), 1.5)
    wrong = lambda p, q: p             # resample from p instead of max(0, p - q)
    first, _ = _lossless_counts(p_logits, q_logits, T, 30000, 3, residual_fn=wrong)
    assert _chi2_p(first, sampling.probs(p_logits[0], T)) < 1e-6


def test_acceptance_rate_is_sum_of_min():
    rng = np.random.default_rng(11)
    V, K, T, n = 12, 1, 0.8, 40000
    p_logits = _rand_logits(rng, (K + 1, V), 2.0)
    q_logits = _rand_logits(rng, (K, V), 2.0)
    p0, q0 = sampling.probs(p_logits[0], T), sampling.probs(q_logits[0], T)
    alpha = float(np.minimum(p0, q0).sum())
    acc = 0
    for _ in range(n):
        d = _draw_drafts([q0], rng.random(1))
        acc += verify(p_logits, q_logits, np.arange(V), d, T, rng.random(1), rng.random()).accept_len
    assert stats.binomtest(acc, n, alpha).pvalue > 1e-4
    assert 0.2 < alpha < 0.9           # the case is not degenerate


def test_q_equal_p_accepts_everything_and_k0_samples_p0():
    rng = np.random.default_rng(12)
    V, K = 8, 4
    tl = _rand_logits(rng, (K + 1, V))
    for _ in range(50):
        drafts = _draw_drafts([sampling.probs(tl[k], 1.0) for k in range(K)], rng.random(K))
        r = verify(tl, tl[:K], np.arange(V), drafts, 1.0, rng.random(K) * 0.999, rng.random())
        assert r.accept_len == K
    # K = 0: the committed token is a plain draw from p_0
    u = 0.37
    r = verify(tl[:1], np.zeros((0, V)), np.arange(V), np.zeros(0, dtype=int), 1.0,
               np.zeros(0), u)
    assert r.accept_len == 0 and r.tokens[0] == sampling.pick_weights(sampling.probs(tl[0], 1.0), u)


def test_unreachable_target_ids_have_zero_q_and_come_from_residual():
    rng = np.random.default_rng(13)
    V_T, V_d = 12, 6
    d2t = np.array([3, 7, -1, 0, 11, 5])
    dl = _rand_logits(rng, V_d)
    dl[d2t < 0] = -np.inf
    q = drafter_probs_on_target(dl, d2t, V_T, 1.0)
    assert abs(q.sum() - 1.0) < 1e-12
    assert np.all(q[[1, 2, 4, 6, 8, 9, 10]] == 0.0)
    # a target that puts all its mass on an unreachable id: every draft is
    # rejected and the residual picks that id
    tl = np.full((2, V_T), -30.0)
    tl[:, 9] = 30.0
    for _ in range(20):
        d = d2t[sampling.pick(dl, 1.0, rng.random())]
        r = verify(tl, dl[None], d2t, np.array([d]), 1.0, rng.random(1), rng.random())
        assert r.accept_len == 0 and r.tokens[0] == 9 and r.residual_used


# ----------------------------------------------------------------------------------------
# Greedy drafting (drafter temperature 0) verified against a sampled target: q is
# one-hot at the drafter's argmax, so the rule reduces to target-only acceptance.
# ----------------------------------------------------------------------------------------
def _greedy_counts(p_logits, q_logits, T, n, seed, T_draft=0.0):
    """Greedy drafts (argmax of each drafter row) verified at target temperature T
    with the drafter temperature T_draft; histograms of the first committed token,
    of the second one when d_0 was accepted, and of the replacement when d_0 was
    rejected, plus the number of accepted d_0."""
    rng = np.random.default_rng(seed)
    K, V = q_logits.shape
    d2t = np.arange(V)
    drafts = np.array([sampling.argmax_lowest(q_logits[k]) for k in range(K)])
    first = np.zeros(V, dtype=np.int64)
    second = np.zeros(V, dtype=np.int64)
    repl = np.zeros(V, dtype=np.int64)
    acc0 = 0
    for _ in range(n):
        r = verify(p_logits, q_logits, d2t, drafts, T, rng.random(K), rng.random(),
                   T_draft=T_draft)
        first[r.tokens[0]] += 1
        if r.accept_len >= 1:
            acc0 += 1
            second[r.tokens[1]] += 1
        else:
            repl[r.tokens[0]] += 1
    return drafts, first, second, repl, acc0


@pytest.mark.parametrize("seed", [0, 1])
def test_greedy_drafting_is_lossless(seed):
    rng = np.random.default_rng(200 + seed)
    V, K, T = 10, 2, 1.0
    p_logits = _rand_logits(rng, (K + 1, V), 1.5)
    q_logits = _rand_logits(rng, (K, V), 1.5)
    _, first, second, _, _ = _greedy_counts(p_logits, q_logits, T, 30000, seed)
    assert _chi2_p(first, sampling.probs(p_logits[0], T)) > 1e-4
    assert _chi2_p(second, sampling.probs(p_logits[1], T)) > 1e-4


def test_greedy_drafting_accepts_with_target_probability_and_redraws_without_draft():
    """Closed forms of the one-hot case: P(accept d_0) = p_0(d_0), and a rejected
    position is redrawn from p_0 with d_0 removed and renormalised."""
    rng = np.random.default_rng(210)
    V, K, T, n = 8, 1, 0.8, 40000
    p_logits = _rand_logits(rng, (K + 1, V), 1.0)
    q_logits = p_logits[:K] + _rand_logits(rng, (K, V), 0.3)   # a drafter close to the target
    drafts, _, _, repl, acc0 = _greedy_counts(p_logits, q_logits, T, n, 5)
    p0 = sampling.probs(p_logits[0], T)
    d = int(drafts[0])
    assert 0.05 < p0[d] < 0.95            # the case is not degenerate
    assert stats.binomtest(acc0, n, p0[d]).pvalue > 1e-4
    expect = p0.copy()
    expect[d] = 0.0
    assert repl[d] == 0
    assert _chi2_p(repl, expect / expect.sum()) > 1e-4


def test_greedy_drafting_test_rejects_sampled_q_for_greedy_drafts():
    """Power check: verifying greedy drafts as if they had been sampled at the
    target's temperature (q = softmax instead of one-hot) is not lossless."""
    rng = np.random.default_rng(220)
    V, K, T = 10, 2, 1.0
    p_logits = _rand_logits(rng, (K + 1, V), 1.5)
    q_logits = _rand_logits(rng, (K, V), 1.5)
    _, first, _, _, _ = _greedy_counts(p_logits, q_logits, T, 30000, 6, T_draft=T)
    assert _chi2_p(first, sampling.probs(p_logits[0], T)) < 1e-6


def test_drafter_temperature_defaults_and_greedy_target():
    """T_draft = None is T_draft = T; a greedy target (T = 0) gives the greedy
    prefix rule whatever the drafter's temperature."""
    rng = np.random.default_rng(230)
    V, K = 9, 4
    d2t = np.arange(V)
    for _ in range(200):
        tl = _rand_logits(rng, (K + 1, V))
        dl = _rand_logits(rng, (K, V))
        drafts = rng.integers(0, V, K)
        j = int(rng.integers(0, K + 1))
        drafts[:j] = np.argmax(tl, axis=1)[:j]        # a matching prefix of random length
        ua, ub = rng.random(K), rng.random()
        for T in (0.0, 0.7):
            a = verify(tl, dl, d2t, drafts, T, ua, ub)
            b = verify(tl, dl, d2t, drafts, T, ua, ub, T_draft=T)
            assert a.accept_len == b.accept_len and np.array_equal(a.tokens, b.tokens)
        g = verify(tl, dl, d2t, drafts, 0.0, ua, ub)
        for Td in (0.0, 1.3):
            x = verify(tl, dl, d2t, drafts, 0.0, ua, ub, T_draft=Td)
            assert x.accept_len == g.accept_len and np.array_equal(x.tokens, g.tokens)
