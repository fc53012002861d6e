"""End-to-end properties of the oracle on the synthetic workloads.

* With the identity vocabulary map and no target noise the target's
  distributions equal the drafter's, so every draft is accepted, at
  temperature 0 (greedy prefix) and above (q = p), and the bonus at T = 0 is
  the target's argmax of the last row.
* Rollback: after each iteration the cached length returns to the
  post-ingest value, and the next ingest carries exactly a + 1 tokens.
* Sequences of one batch are independent (running b alone or after others
  gives the same result).
"""
import numpy as np

import synth
from oracle import harness


def test_noise_free_identity_target_accepts_every_draft():
    base = synth.get("p_qwen_small").with_(name="nf", cfg_id=201, sigma=0.0, n_layers=1,
                                            vocab_draft=501, vocab_target=501, temps=(0.0, 1.0))
    for b in range(2):
        its = harness.run_sequence(base, b, 3)
        for it in its:
            assert it.result.accept_len == base.K
            if base.temperature(b) == 0.0:
                assert it.result.tokens[base.K] == int(np.argmax(it.target_logits[base.K]))


def test_rollback_and_ingest_lengths():
    w = synth.get("p_partial")
    its = harness.run_sequence(w, 1, 4)
    for prev, cur in zip(its, its[1:]):
        assert cur.pre_len == prev.committed
        assert len(cur.new_tokens) == prev.result.accept_len + 1
        assert cur.committed == cur.pre_len + len(cur.new_tokens)
        assert list(cur.new_tokens) == list(prev.result.tokens[: prev.result.accept_len + 1])


def test_sequences_are_independent():
    w = synth.get("p_inject")
    a = harness.run_sequence(w, 1, 2)
    dr = harness.build_drafter(w)
    harness.run_sequence(w, 0, 2, drafter=dr)
    b = harness.run_sequence(w, 1, 2, drafter=dr)
    for x, y in zip(a, b):
        assert np.array_equal(x.drafts, y.drafts)
        assert np.array_equal(x.draft_logits, y.draft_logits)
        assert x.result.accept_len == y.result.accept_len
