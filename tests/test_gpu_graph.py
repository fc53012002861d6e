"""osprey_graph_*: one steady-state iteration (pending draft call + verification)
captured as a HIP graph over fixed buffers and replayed.

Every replay must give bit-for-bit the results of the same iteration launched call
by call (the kernels and their order are the same), with the program's own eager
work (copying the next iteration's inputs into the captured buffers) between
replays.  The host state must advance as the two calls would, and misuse must be
refused before anything is enqueued."""
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


def _say(*a):
    print(*a, flush=True)


def _reference(w, n_it):
    """Stream launches: per iteration the inputs, the target logits and the outputs."""
    from paper_2609_09338_amd import workload as WL
    s = WL.make_drafter(w, n_it)
    WL.reset_sequences(s)
    out = WL.alloc_outputs(s)
    rec = []
    for it in range(n_it):
        inp = WL.iter_inputs(s, it)
        WL.draft(s, it, inp, out)
        tl = WL.synthetic_target(s, it, out.logits)
        WL.verify(s, inp, tl, out)
        torch.cuda.synchronize()
        rec.append((inp, tl, [t.clone() for t in (out.drafts, out.logits, out.accept_len,
                                                   out.mask, out.tokens)]))
    return s, out, rec


@pytest.mark.parametrize("name", ["p_qwen_small", "p_single128", "p_block"])
def test_graph_replays_equal_stream_launches(name):
    _require_gpu()
    from paper_2609_09338_amd import workload as WL
    w = synth.get(name)
    n_it = 5
    _say(f"[graph] {name}: stream reference")
    s, out, rec = _reference(w, n_it)
    B = w.batch
    # back to the start, on a stream of its own, iteration 0 (explicit) call by call
    st = torch.cuda.Stream()
    s.drafter.set_stream(st)
    for b in range(B):
        s.drafter.seq_truncate(b, int(s.ctx[b]) - 1)
    inp0, tl0, _ = rec[0]
    WL.draft(s, 0, inp0, out)
    WL.verify(s, inp0, tl0, out)
    # fixed input buffers the graph reads
    fx_taps = torch.empty_like(inp0.taps)
    fx_ud, fx_ua, fx_ub = (torch.empty_like(inp0.u_draft), torch.empty_like(inp0.u_accept),
                           torch.empty_like(inp0.u_bonus))
    fx_tl = torch.empty_like(tl0)
    mask = synth.mask_token(w) if w.drafting == "block" else None
    _say(f"[graph] {name}: capture")
    g = s.drafter.capture_iteration(list(range(B)), w.K, fx_taps, s.draft_temperature, fx_ud,
                                    out.drafts, out.logits, fx_tl, s.temperature, fx_ua, fx_ub,
                                    out.accept_len, out.mask, out.tokens,
                                    max_context=int(s.drafter.cfg.max_seq_len),
                                    taps_stride=w.K + 1, mask_token=mask)
    for it in range(1, n_it):
        inp, tl, ref = rec[it]
        with torch.cuda.stream(st):
            for dst, src in ((fx_taps, inp.taps), (fx_ud, inp.u_draft), (fx_ua, inp.u_accept),
                             (fx_ub, inp.u_bonus), (fx_tl, tl)):
                dst.copy_(src)
        g.launch()
        st.synchronize()
        _say(f"[graph] {name}: replay {it}")
        for got, want in zip((out.drafts, out.logits, out.accept_len, out.mask, out.tokens), ref):
            assert torch.equal(got, want), (name, it)
    assert s.drafter.device_errors() == 0
    # the host state advanced as the calls would: the next call-by-call iteration is allowed
    # and lands where the recorded trajectory says
    lengths = [s.drafter.seq_length(b) for b in range(B)]
    want = [int(s.ctx[b]) + sum(int(rec[j][2][2][b]) + 1 for j in range(n_it - 1))
            for b in range(B)]
    assert lengths == want, (lengths, want)
    g.close()


def test_graph_misuse_is_refused():
    _require_gpu()
    from paper_2609_09338_amd import _lib as L
    from paper_2609_09338_amd import workload as WL
    from paper_2609_09338_amd.binding import OspreyError
    w = synth.get("p_single128")
    s, out, rec = _reference(w, 2)
    inp, tl, _ = rec[1]
    args = ([0], w.K, inp.taps, s.draft_temperature, inp.u_draft, out.drafts, out.logits, tl,
            s.temperature, inp.u_accept, inp.u_bonus, out.accept_len, out.mask, out.tokens)
    kw = dict(max_context=int(s.drafter.cfg.max_seq_len), taps_stride=w.K + 1)

    def code(fn):
        with pytest.raises(OspreyError) as e:
            fn()
        return e.value.status

    # the null stream cannot be captured
    assert code(lambda: s.drafter.capture_iteration(*args, **kw)) == L.OSPREY_E_INVALID
    st = torch.cuda.Stream()
    s.drafter.set_stream(st)
    # kernel timing on
    s.drafter.kernel_timing((0,))
    assert code(lambda: s.drafter.capture_iteration(*args, **kw)) == L.OSPREY_E_STATE
    s.drafter.kernel_timing(())
    # a context bound the slot already exceeds
    assert code(lambda: s.drafter.capture_iteration(*args, max_context=8,
                                                    taps_stride=w.K + 1)) == L.OSPREY_E_CAPACITY
    g = s.drafter.capture_iteration(*args, **kw)
    # capturing ran nothing and changed no state: the slot is still VERIFIED and a
    # call-by-call iteration still works
    WL.draft(s, 1, inp, out)
    # DRAFTED now: a graph launch needs VERIFIED slots
    assert code(g.launch) == L.OSPREY_E_STATE
    WL.verify(s, inp, tl, out)
    g.launch()
    st.synchronize()
    assert s.drafter.device_errors() == 0
    g.close()
