"""Run the synthetic workloads through the oracle, one sequence at a time.

Sequences of a batch never interact (each has its own cache, tokens and
uniforms), so any subset of a batch can be reproduced on its own.

Per sequence b:
* positions [0, ctx-1) are filled first: with synthetic post-RoPE keys and
  values ("kv" workloads) or by ingesting the first ctx-1 prompt tokens with
  zero drafts ("ingest" workloads; the row of position 0 has zero taps);
* iteration 0 ingests prompt token ctx-1; iteration i > 0 ingests the a+1
  tokens committed by iteration i-1; the conditioning rows are the first
  n_new rows of `synth.taps(w, i, b, K + 1)`;
* K drafts are proposed (a chain of K steps, or one block for workloads that
  draft in blocks), the synthetic target logits are formed from the drafter's
  logits (`synth.target_logits`), and verify decides.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Dict, List, Optional

import numpy as np

import synth
from .block import draft_block
from .drafter import Drafter, Sequence
from .verify import VerifyResult, verify


@dataclass
class Iteration:
    pre_len: int                # cached length before the ingest
    new_tokens: np.ndarray      # tokens ingested this iteration
    committed: int              # cached length after the ingest
    drafts: np.ndarray          # [K] target ids
    draft_rows: np.ndarray      # [K] LM-head rows sampled
    draft_logits: np.ndarray    # [K, V_d]
    target_logits: np.ndarray   # [K + 1, V_T] float32 (the synthetic input to verify)
    result: VerifyResult


def build_drafter(w, weights=None, d2t=None) -> Drafter:
    weights = synth.make_weights(w) if weights is None else weights
    d2t = synth.make_d2t(w) if d2t is None else d2t
    return Drafter(w, weights, d2t)


def start_sequence(w, drafter: Drafter, b: int, n_iters: int) -> Sequence:
    ctx = int(synth.context_lengths(w)[b])
    seq = Sequence(w, ctx + (n_iters + 1) * (w.K + 1) + 1)
    if w.prefill == "kv":
        k, v = synth.context_kv(w, b, ctx - 1)
        seq.k[:, : ctx - 1] = k
        seq.v[:, : ctx - 1] = v
        seq.length = ctx - 1
    else:
        prompt = synth.prompt_tokens(w, b, ctx)
        if ctx > 1:
            taps = synth.taps(w, -1, b, ctx - 1).astype(np.float64)
            taps[0] = 0.0
            drafter.ingest(seq, prompt[: ctx - 1], taps)
    return seq


def run_sequence_timed(w, b: int, n_max: int, seconds: float,
                       drafter: Optional[Drafter] = None) -> List[Iteration]:
    """Iterations of sequence b until `seconds` have elapsed (at least one); the
    records keep no logit rows (a long timed run would otherwise hold gigabytes)."""
    import time
    t0 = time.perf_counter()
    return run_sequence(w, b, n_max, drafter=drafter,
                        stop=lambda: time.perf_counter() - t0 > seconds, lean=True)


def run_sequence(w, b: int, n_iters: int, drafter: Optional[Drafter] = None,
                 residual_fn=None, stop=None, lean: bool = False) -> List[Iteration]:
    drafter = drafter or build_drafter(w)
    seq = start_sequence(w, drafter, b, n_iters)
    ctx = int(synth.context_lengths(w)[b])
    new_tokens = synth.prompt_tokens(w, b, ctx)[ctx - 1:ctx].astype(np.int64)
    T = w.temperature(b)
    Td = w.draft_temperature(b)
    out = []
    for it in range(n_iters):
        pre = seq.length
        taps = synth.taps(w, it, b, w.K + 1)[: len(new_tokens)]
        ud = synth.u_draft(w, it)[b]
        if w.drafting == "block":
            drafts, logits, rows, committed = draft_block(drafter, seq, new_tokens, taps, w.K, Td,
                                                          ud, synth.mask_token(w))
        else:
            drafts, logits, rows, committed = drafter.draft(seq, new_tokens, taps, w.K, Td, ud)
        tl = synth.target_logits(w, logits, drafter.d2t, synth.target_noise(w, it, b))
        res = verify(tl, logits, drafter.d2t, drafts, T, synth.u_accept(w, it)[b],
                     float(synth.u_bonus(w, it)[b]), residual_fn=residual_fn, T_draft=Td)
        out.append(Iteration(pre, new_tokens.copy(), committed, drafts, rows,
                             None if lean else logits, None if lean else tl, res))
        drafter.rollback(seq, committed)
        new_tokens = res.tokens[: res.accept_len + 1].copy()
        if stop is not None and stop():
            break
    return out
