"""Many-draw check of the acceptance rule on the HIP path (the standard rule of
Section 3.1, whose losslessness the paper relies on, Section 1).

osprey_verify_rows decides 102400 sequences of a 24-token vocabulary (400 calls of
256), every one with the same target rows p and drafter rows q and its own uniforms,
drafts drawn from q (or greedy, q one-hot).  Every decision -- each acceptance, the
accepted length, the resampled or bonus token -- must equal the oracle's bit for bit,
except draws inside the flag windows (a uniform within 1e-5 of its ratio; both sides
read the same logits), and the first committed token must follow p_0 (chi-square,
p > 1e-4), the second, given the first draft accepted, p_1."""
import numpy as np
import pytest
import torch
from scipy import stats

import synth
from oracle import sampling as OS
from oracle.verify import verify as o_verify

from . import parity

pytestmark = pytest.mark.gpu

V, K, B, CALLS = 24, 2, 256, 400


def _require_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_09338_amd import _lib
    _lib.load()


@pytest.mark.parametrize("dmode", ["sampled", "greedy"])
def test_acceptance_rule_over_many_draws(dmode):
    _require_gpu()
    from paper_2609_09338_amd import workload as WL
    print(f"[acceptance] {dmode}: {CALLS} calls of {B}", flush=True)
    w = synth.Workload(name=f"acc_{dmode}", cfg_id=350, dtype="bf16", n_layers=1, d_model=64,
                       n_q_heads=1, n_kv_heads=1, head_dim=64, d_ffn=64, vocab_draft=V,
                       vocab_target=V, target_hidden=8, batch=B, K=K, ctx_lo=1, ctx_hi=1)
    s = WL.make_drafter(w, 1)
    d2t = np.arange(V)
    rng = np.random.default_rng(2609 + (dmode == "greedy"))
    tl1 = (rng.standard_normal((K + 1, V)) * 1.5).astype(np.float32)
    dl1 = (rng.standard_normal((K, V)) * 1.5).astype(np.float32)
    T, Td = 1.0, (1.0 if dmode == "sampled" else 0.0)
    dev = s.device
    tl = torch.from_numpy(np.ascontiguousarray(np.broadcast_to(tl1, (B, K + 1, V)))).to(dev)
    dl = torch.from_numpy(np.ascontiguousarray(np.broadcast_to(dl1, (B, K, V)))).to(dev)
    temp = torch.full((B,), T, dtype=torch.float32, device=dev)
    temp_d = torch.full((B,), Td, dtype=torch.float32, device=dev)
    al = torch.empty(B, dtype=torch.int32, device=dev)
    mk = torch.empty((B, K), dtype=torch.uint8, device=dev)
    ot = torch.empty((B, K + 1), dtype=torch.int32, device=dev)
    # drafts follow q: inverse CDF over the drafter row (greedy: its argmax)
    w_q = [OS.softmax_weights(dl1[k], Td) if Td > 0 else None for k in range(K)]
    cdf_q = [np.cumsum(x) if x is not None else None for x in w_q]
    first, second = np.zeros(V, dtype=np.int64), np.zeros(V, dtype=np.int64)
    flagged = accepted0 = 0
    for c in range(CALLS):
        u_d = rng.integers(0, 1 << 24, (B, K)) * 2.0 ** -24
        if Td > 0:
            drafts = np.stack([np.searchsorted(cdf_q[k], u_d[:, k] * cdf_q[k][-1], side="right")
                               for k in range(K)], axis=1).astype(np.int32)
        else:
            drafts = np.tile(np.argmax(dl1, axis=1).astype(np.int32), (B, 1))
        u_a = (rng.integers(0, 1 << 24, (B, K)) * 2.0 ** -24).astype(np.float32)
        u_b = (rng.integers(0, 1 << 24, B) * 2.0 ** -24).astype(np.float32)
        f = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
        s.drafter.verify_rows(K, tl, dl, f(drafts), temp, f(u_a), f(u_b), al, mk, ot,
                              draft_temperature=temp_d)
        torch.cuda.synchronize()
        g_a, g_m, g_t = al.cpu().numpy(), mk.cpu().numpy(), ot.cpu().numpy()
        for b in range(B):
            r = o_verify(tl1, dl1, d2t, drafts[b], T, u_a[b], float(u_b[b]), T_draft=Td)
            same = (g_a[b] == r.accept_len and np.array_equal(g_m[b], r.mask)
                    and np.array_equal(g_t[b], r.tokens))
            if not same:
                assert parity.verify_flags(r, tl1, dl1, d2t, drafts[b], T, u_a[b], float(u_b[b]),
                                           T_draft=Td), (dmode, c, b, g_a[b], r.accept_len,
                                                         g_t[b], r.tokens)
                flagged += 1
        first += np.bincount(g_t[:, 0], minlength=V)
        ok0 = g_a >= 1
        accepted0 += int(ok0.sum())
        second += np.bincount(g_t[ok0, 1], minlength=V)
    assert s.drafter.device_errors() == 0
    n = CALLS * B
    p0 = OS.probs(tl1[0], T)
    p1 = OS.probs(tl1[1], T)
    pv0 = stats.chisquare(first, n * p0).pvalue
    pv1 = stats.chisquare(second, accepted0 * p1).pvalue
    print(f"[acceptance] {dmode}: {n} sequences, {flagged} flagged, first-token chi2 p={pv0:.3g}, "
          f"second-token chi2 p={pv1:.3g} over {accepted0}", flush=True)
    assert flagged <= n // 1000
    assert pv0 > 1e-4 and pv1 > 1e-4
