"""CPU oracle for the Osprey draft-and-verify step -- TEST INFRASTRUCTURE ONLY.

A plain, slow, obviously correct numpy implementation (float64 arithmetic)
of what the GPU path computes:

* `drafter`  -- the converted drafter of Section 3.3: target hidden-state tap
  projection (Eq. 1), zero-initialised QKV expansion (Eq. 2-3), a pre-norm
  decoder body transferred unchanged from the pruned source LM (Section 3.2,
  Stage 1), final norm and the vocabulary-aligned LM head, run token by token
  over its own KV cache, with the drafter's own last hidden state fed back as
  the conditioning input at draft steps (Section 3.4).
* `sampling` -- the rule that turns logits and a uniform into a token.
* `verify`   -- the standard speculative-decoding acceptance rule the paper
  keeps unchanged (Section 3.1): greedy prefix match at temperature 0,
  min(1, p/q) acceptance with residual resampling otherwise.
* `harness`  -- runs the synthetic workloads through the above.

Only `tests/`, `__graft_entry__.smoke()` and the CPU-baseline leg of
`bench.py` may import this package.  It shares no code with the HIP path;
both read their inputs from `synth`, which holds no arithmetic of the method.

Parity pins (tests/test_oracle_*.py): the zero-expansion drafter equals an
independent library decoder (transformers' Qwen3); a constant conditioning
input equals that decoder with Q/K/V biases; RoPE relativity, attention
special cases, bf16 rounding against torch, sampling against searchsorted,
greedy prefix by construction, losslessness by chi-square, acceptance rate
against sum(min(p, q)), and parameter counts against the paper's table of
draft sizes.  Parity unpinned: whether the fed-back hidden state is taken
before or after the final norm (the paper does not say; the pre-norm
residual is used).
"""
