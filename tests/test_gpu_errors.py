"""Error paths of the draft-tree and block entry points on the GPU: invalid arguments
are refused before anything is enqueued (status code, nothing written, the slots'
state unchanged), and a valid call afterwards runs and verifies as if nothing had
happened (against the same call on a drafter that never saw the bad ones)."""
import numpy as np
import pytest
import torch

import synth

pytestmark = pytest.mark.gpu


def _require_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_09338_amd import _lib
    _lib.load()


def _setup():
    from paper_2609_09338_amd import workload as WL
    w = synth.PARITY["p_block"]
    s = WL.make_drafter(w, 2)
    WL.reset_sequences(s)
    return w, s, WL


def _block(s, w, WL, inp, out, K=None, mask=None):
    slots = list(range(w.batch))
    s.drafter.draft_step(slots, w.K if K is None else K, inp.taps, s.draft_temperature,
                         inp.u_draft, n_new=[1] * w.batch, new_tokens=inp.new_tokens,
                         taps_stride=w.K + 1, draft_tokens=out.drafts, draft_logits=out.logits,
                         mask_token=synth.mask_token(w) if mask is None else mask)


def test_invalid_block_and_tree_calls_change_nothing():
    _require_gpu()
    from paper_2609_09338_amd import _lib as L
    from paper_2609_09338_amd.binding import OspreyError
    print("[errors] p_block", flush=True)
    w, s, WL = _setup()
    inp = WL.iter_inputs(s, 0)
    out = WL.alloc_outputs(s)
    out.drafts.fill_(-7)
    dev, B = s.device, w.batch
    for kw in (dict(K=1), dict(mask=-1), dict(mask=w.vocab_target)):
        with pytest.raises(OspreyError) as e:
            _block(s, w, WL, inp, out, **kw)
        assert e.value.status == L.OSPREY_E_INVALID, kw
    # more proposals than max_k (buffers sized for them)
    K1 = w.K + 1
    d1 = torch.full((B, K1), -7, dtype=torch.int32, device=dev)
    with pytest.raises(OspreyError) as e:
        s.drafter.draft_step(list(range(B)), K1, inp.taps, s.draft_temperature,
                             torch.zeros((B, K1), dtype=torch.float32, device=dev),
                             n_new=[1] * B, new_tokens=inp.new_tokens, taps_stride=w.K + 1,
                             draft_tokens=d1,
                             draft_logits=torch.zeros((B, K1, w.vocab_draft), device=dev),
                             mask_token=synth.mask_token(w))
    assert e.value.status == L.OSPREY_E_INVALID
    tk = torch.full((B, 8), -7, dtype=torch.int32, device=dev)
    pr = torch.full((B, 8), -7, dtype=torch.int32, device=dev)
    taps = inp.taps
    for topk, depth, n in ((1, 3, 3), (w.K + 1, 2, 8), (2, 0, 2), (2, 9, 8), (2, 2, 7), (2, 2, 0)):
        with pytest.raises(OspreyError) as e:
            s.drafter.draft_tree(list(range(B)), topk, depth, n, taps, s.temperature,
                                 tk, pr,
                                 n_new=[1] * B, new_tokens=inp.new_tokens, taps_stride=w.K + 1)
        assert e.value.status == L.OSPREY_E_INVALID, (topk, depth, n)
    # verify with nothing drafted: a state error
    tl = torch.zeros((B, w.K + 1, w.vocab_target), dtype=torch.float32, device=dev)
    with pytest.raises(OspreyError) as e:
        WL.verify(s, inp, tl, out)
    assert e.value.status == L.OSPREY_E_STATE
    torch.cuda.synchronize()
    assert (out.drafts == -7).all() and (d1 == -7).all() and (tk == -7).all() and (pr == -7).all()
    for b in range(B):
        assert s.drafter.seq_length(b) == int(s.ctx[b]) - 1
    # a valid block afterwards equals the same block on a fresh drafter
    _block(s, w, WL, inp, out)
    w2, s2, _ = _setup()
    out2 = WL.alloc_outputs(s2)
    _block(s2, w2, WL, WL.iter_inputs(s2, 0), out2)
    torch.cuda.synchronize()
    assert torch.equal(out.drafts, out2.drafts)
    assert torch.equal(out.logits, out2.logits)
    assert s.drafter.device_errors() == 0 and s2.drafter.device_errors() == 0
