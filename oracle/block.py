"""Block drafting with the EAGLE-style target interface of the DFlash ablation (test
infrastructure: only tests, the smoke check and the benchmark's CPU baseline call
this module).

The appendix on DFlash drafts a block of B positions in one forward pass: the last
verified token (the anchor) followed by B - 1 mask placeholders.  In its EAGLE-style
variant every attention layer keeps the drafter's own projections and adds
zero-initialised target-side ones (the expanded QKV of Eq. 2-3), the target feature
is taken once at the anchor and broadcast to every position of the block, the
block's attention is the drafter's causal self-attention, and position k of the
block predicts the token at k + 1.

So for K proposals (a block of K + 1 positions; the last mask predicts past the
block and is not needed under causal attention):

  the committed tokens are ingested as usual, the anchor last (its row's
  conditioning input s_a is the projected taps of the position before it);
  mask rows j = 1 .. K - 1 run at positions committed + j - 1 with the mask token
  and s_a as their conditioning input, attending causally to the cache (the
  context, the anchor and the earlier masks);
  proposal k is drawn from the logits of block row k (row 0: the anchor) at the
  drafter temperature with uniform u_k, independently of the other proposals.

The mask rows' cache entries lie past the committed length and are rolled back
with the rest of the draft.  The proposals are verified with the ordinary chain
rule: each was drawn from its row's distribution q_k, which does not depend on
the other proposals, so accepting with min(1, p_k / q_k) and resampling the
residual stays lossless."""
from __future__ import annotations

import numpy as np

from . import sampling


def draft_block(drafter, seq, tokens, taps, K: int, T: float, u_draft, mask_token: int):
    """Ingest the committed tokens, then propose K drafts from one block.

    Returns (drafts [K] target ids, logits [K, V_d], draft_rows [K],
    committed_length), like the chain's draft."""
    s_rows = drafter.project_taps(taps)
    g = drafter.ingest(seq, tokens, taps)
    committed = seq.length
    s_anchor = s_rows[-1]
    outs = [g]
    for j in range(1, K):
        outs.append(drafter.forward_row(seq, int(mask_token), s_anchor, committed + j - 1))
    drafts, rows, logit_rows = [], [], []
    for k in range(K):
        l = drafter.logits(outs[k])
        r = sampling.pick(l, T, float(u_draft[k]))
        rows.append(r)
        drafts.append(int(drafter.d2t[r]))
        logit_rows.append(l)
    L = np.stack(logit_rows) if K else np.zeros((0, drafter.cfg.vocab_draft))
    return np.array(drafts, dtype=np.int64), L, np.array(rows, dtype=np.int64), committed
