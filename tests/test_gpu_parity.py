"""GPU parity: the HIP path through the C ABI against the CPU oracle.

* verify_rows on synthetic inputs (identical drafter and target logits on both
  sides): accepted lengths, masks and tokens bit-exact except flagged
  near-threshold decisions;
* whole draft -> verify iterations on the parity workloads (ragged
  vocabularies, partial and injective vocabulary maps, shuffled KV pages,
  contexts straddling page boundaries, greedy and sampled requests in one
  batch), chains and blocks (the anchor and mask rows of block drafting, a
  Llama-shaped body without QK-norm): drafter logits within 2e-2 (bf16) / 1e-4
  (fp32), draft ids and verification outcomes bit-exact unless flagged (see
  tests/parity.py);
* the zero-initialised expansion (Eq. 3) on the GPU: logits independent of the
  taps, bit for bit.
"""
import numpy as np
import pytest
import torch

import synth
from oracle import harness as OH
from oracle import sampling as OS
from oracle.verify import verify as o_verify

from . import parity

pytestmark = pytest.mark.gpu


def _require_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_09338_amd import _lib
    _lib.load()


def _say(*a):
    print(*a, flush=True)


# ----------------------------------------------------------------------------------------
# verify_rows: same inputs on both sides
# ----------------------------------------------------------------------------------------
@pytest.mark.parametrize("name,V_d,V_T,vmap,dmode", [
    ("small_partial", 997, 811, "partial", "same"),
    ("inject", 3001, 4513, "inject", "same"),
    ("large_identity", 151936, 151936, "identity", "same"),
    ("small_partial_greedy_draft", 997, 811, "partial", "mixed"),
    ("inject_greedy_draft", 3001, 4513, "inject", "mixed"),
    ("large_identity_greedy_draft", 151936, 151936, "identity", "greedy")])
def test_verify_rows_matches_oracle(name, V_d, V_T, vmap, dmode):
    """dmode: drafts drawn at the target's temperature ("same"), greedily ("greedy":
    q one-hot, target-only acceptance) or at a mix of greedy, equal and other
    drafter temperatures ("mixed")."""
    _require_gpu()
    from paper_2609_09338_amd import workload as WL
    _say(f"[verify_rows] {name}")
    w = synth.Workload(name=f"vr_{name}", cfg_id=300 + V_d % 97, dtype="bf16", n_layers=1,
                       d_model=64, n_q_heads=1, n_kv_heads=1, head_dim=64, d_ffn=64,
                       vocab_draft=V_d, vocab_target=V_T, target_hidden=8, batch=16, K=5,
                       ctx_lo=1, ctx_hi=1, vocab_map=vmap)
    s = WL.make_drafter(w, 1)
    d2t = synth.make_d2t(w)
    rng = np.random.default_rng(42)
    B, K = w.batch, w.K
    temps = np.array([[0.0, 0.7, 1.0, 1.3][b % 4] for b in range(B)], dtype=np.float32)
    if dmode == "same":
        temps_d = temps.copy()
    elif dmode == "greedy":
        temps_d = np.zeros(B, dtype=np.float32)
    else:
        temps_d = np.array([[0.0, 0.0, 1.0, 0.5][(b // 2) % 4] for b in range(B)],
                           dtype=np.float32)
    sig = np.array([[0.05, 0.5, 1.0, 3.0][(b // 4) % 4] for b in range(B)])
    dl = (rng.standard_normal((B, K, V_d)) * 1.5).astype(np.float32)
    dl[:, :, d2t < 0] = -np.inf
    u_d = rng.integers(0, 1 << 24, (B, K)) * 2.0 ** -24
    drafts = np.zeros((B, K), dtype=np.int32)
    for b in range(B):
        for k in range(K):
            drafts[b, k] = d2t[OS.pick(dl[b, k], float(temps_d[b]), float(u_d[b, k]))]
    noise = rng.standard_normal((B, K + 1, V_T)).astype(np.float32)
    tl = np.zeros((B, K + 1, V_T), dtype=np.float32)
    for b in range(B):
        wb = w.with_(sigma=float(sig[b]))
        tl[b] = synth.target_logits(wb, dl[b], d2t, noise[b])
    u_a = (rng.integers(0, 1 << 24, (B, K)) * 2.0 ** -24).astype(np.float32)
    u_b = (rng.integers(0, 1 << 24, B) * 2.0 ** -24).astype(np.float32)
    dev = s.device
    T = lambda a, dt=None: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    al = torch.empty(B, dtype=torch.int32, device=dev)
    mk = torch.empty((B, K), dtype=torch.uint8, device=dev)
    ot = torch.empty((B, K + 1), dtype=torch.int32, device=dev)
    s.drafter.verify_rows(K, T(tl), T(dl), T(drafts), T(temps), T(u_a), T(u_b), al, mk, ot,
                          draft_temperature=None if dmode == "same" else T(temps_d))
    torch.cuda.synchronize()
    assert s.drafter.device_errors() == 0
    al, mk, ot = al.cpu().numpy(), mk.cpu().numpy(), ot.cpu().numpy()
    flagged = 0
    accepted = 0
    for b in range(B):
        r = o_verify(tl[b], dl[b], d2t, drafts[b], float(temps[b]), u_a[b], float(u_b[b]),
                     T_draft=float(temps_d[b]))
        same = (al[b] == r.accept_len and np.array_equal(mk[b], r.mask)
                and np.array_equal(ot[b], r.tokens))
        if not same:
            assert parity.verify_flags(r, tl[b], dl[b], d2t, drafts[b], float(temps[b]), u_a[b],
                                       float(u_b[b]), T_draft=float(temps_d[b])), \
                (b, al[b], r.accept_len, ot[b], r.tokens)
            flagged += 1
        accepted += r.accept_len
    assert flagged <= 2
    assert accepted > 0


# ----------------------------------------------------------------------------------------
# whole iterations
# ----------------------------------------------------------------------------------------
def _delta(gl: np.ndarray, ol: np.ndarray) -> float:
    m = np.isfinite(ol)
    assert np.array_equal(m, np.isfinite(gl)), "masked rows differ"
    return float(np.max(np.abs(gl[m].astype(np.float64) - ol[m]))) if m.any() else 0.0


def _run_parity(w, n_iters, seqs, tol):
    """Run every sequence of w on the GPU; compare the sampled `seqs` with the oracle."""
    from paper_2609_09338_amd import workload as WL
    _say(f"[parity] {w.name}: oracle for sequences {seqs}")
    dr_o = OH.build_drafter(w)
    ref = {b: OH.run_sequence(w, b, n_iters, drafter=dr_o) for b in seqs}
    d2t = dr_o.d2t
    _say(f"[parity] {w.name}: GPU")
    s = WL.make_drafter(w, n_iters)
    WL.reset_sequences(s)
    out = WL.alloc_outputs(s)
    live = set(seqs)
    # exact_*: comparisons that were made and came out equal, unflagged -- draft ids,
    # acceptance decisions (one per draft the rule tested) and the resampled / bonus token
    stats = dict(compared=0, flagged=0, max_delta=0.0, accepted=0, exact_drafts=0,
                 exact_accepts=0, exact_bonus=0)
    for it in range(n_iters):
        inp = WL.iter_inputs(s, it)
        WL.draft(s, it, inp, out)
        torch.cuda.synchronize()
        g_logits = out.logits.cpu().numpy()
        g_drafts = out.drafts.cpu().numpy()
        synth_rows = WL.synthetic_target(s, it, out.logits, d2t)
        for b in live:
            synth_rows[b] = torch.from_numpy(ref[b][it].target_logits).to(s.device)
        WL.verify(s, inp, synth_rows.contiguous(), out)
        torch.cuda.synchronize()
        g_a, g_mask, g_tok = (out.accept_len.cpu().numpy(), out.mask.cpu().numpy(),
                              out.tokens.cpu().numpy())
        for b in sorted(live):
            rec = ref[b][it]
            T, Td = w.temperature(b), w.draft_temperature(b)
            ok = True
            for k in range(w.K):
                delta = _delta(g_logits[b, k], rec.draft_logits[k])
                stats["max_delta"] = max(stats["max_delta"], delta)
                assert delta <= tol, (w.name, b, it, k, delta)
                if g_drafts[b, k] != rec.drafts[k]:
                    u = float(synth.u_draft(w, it)[b, k])
                    assert parity.draw_flag(rec.draft_logits[k], Td, u, delta), \
                        (w.name, b, it, k, g_drafts[b, k], rec.drafts[k])
                    ok = False
                    break
                stats["exact_drafts"] += 1
            if ok:
                same = (g_a[b] == rec.result.accept_len and
                        np.array_equal(g_mask[b], rec.result.mask) and
                        np.array_equal(g_tok[b], rec.result.tokens))
                if same:
                    # decisions tested: the a accepted drafts, plus the rejection if a < K
                    stats["exact_accepts"] += int(rec.result.accept_len) + \
                        int(rec.result.accept_len < w.K)
                    stats["exact_bonus"] += 1
                else:
                    delta = max(_delta(g_logits[b, k], rec.draft_logits[k]) for k in range(w.K))
                    assert parity.verify_flags(rec.result, rec.target_logits, rec.draft_logits,
                                               d2t, rec.drafts, T, synth.u_accept(w, it)[b],
                                               float(synth.u_bonus(w, it)[b]), delta, T_draft=Td), \
                        (w.name, b, it, g_a[b], rec.result.accept_len, g_tok[b], rec.result.tokens)
                    ok = False
            stats["compared"] += 1
            stats["accepted"] += int(rec.result.accept_len)
            if not ok:
                stats["flagged"] += 1
                live.discard(b)
    assert s.drafter.device_errors() == 0
    _say(f"[parity] {w.name}: {stats}")
    assert stats["flagged"] <= max(1, stats["compared"] // 5), stats
    return stats


def _assert_exact_comparisons(stats, name):
    """A case passes on flags alone only if nothing was compared exactly: require at
    least one unflagged draft id, acceptance decision and resampled / bonus token."""
    for key in ("exact_drafts", "exact_accepts", "exact_bonus"):
        assert stats[key] >= 1, (name, key, stats)


@pytest.mark.parametrize("name", ["p_tiny_f32", "p_qwen_small", "p_partial", "p_inject",
                                  "p_greedy_draft", "p_single64", "p_single128", "p_single_splits",
                                  "p_single_splits64", "p_block", "p_block_single", "p_wide_taps"])
def test_iterations_match_oracle(name):
    _require_gpu()
    w = synth.get(name)
    tol = 1e-4 if w.dtype == "f32" else 2e-2
    _run_parity(w, 4, list(range(w.batch)), tol)


@pytest.mark.parametrize("name,K", [("p_single64", 2), ("p_single64", 3), ("p_partial", 2),
                                    ("p_partial", 3), ("p_qwen_small", 3)])
def test_short_chains_match_oracle(name, K):
    """Chains of two and three drafts: where each draft is drawn (a single sequence: the
    next step's QKV GEMV but for the last; batches: the sampling kernel for the first and
    last, the next step's row preparation between) at the shortest chains."""
    _require_gpu()
    w = synth.get(name).with_(name=f"{name}_K{K}", K=K)
    tol = 1e-4 if w.dtype == "f32" else 2e-2
    _run_parity(w, 3, list(range(w.batch)), tol)


def test_tiny_fp32_variants_match_oracle():
    """The small fp32 chain draft: zero and N(0, 0.02) expansion, greedy and T = 1,
    noise sigma 0.5 and 2 (8 runs)."""
    _require_gpu()
    base = synth.get("c1")
    v = 0
    for exp in ("zero", "normal"):
        for T in (0.0, 1.0):
            for sig in (0.5, 2.0):
                v += 1
                w = base.with_(name=f"c1_v{v}", variant=v, expansion=exp, temps=(T,), sigma=sig)
                _run_parity(w, 3, [0], 1e-4)


def test_zero_expansion_ignores_taps_bitwise():
    """Eq. 3 on the GPU: with zero c-slot columns the drafter's logits and drafts
    do not depend on the target taps (0 * x is exact for finite x)."""
    _require_gpu()
    from paper_2609_09338_amd import workload as WL
    w = synth.get("p_qwen_small").with_(name="zero_exp", cfg_id=41, expansion="zero")
    res = []
    for scale in (1.0, 0.0):
        s = WL.make_drafter(w, 1)
        WL.reset_sequences(s)
        out = WL.alloc_outputs(s)
        inp = WL.iter_inputs(s, 0)
        inp.taps.mul_(scale)
        WL.draft(s, 0, inp, out)
        torch.cuda.synchronize()
        res.append((out.logits.cpu().numpy().copy(), out.drafts.cpu().numpy().copy()))
    assert np.array_equal(res[0][0], res[1][0])
    assert np.array_equal(res[0][1], res[1][1])


def test_runs_are_deterministic_and_page_order_free():
    """Two runs give bit-identical results, and so does a different physical page
    assignment of the same sequences (the cache is addressed through the block table)."""
    _require_gpu()
    from paper_2609_09338_amd import workload as WL
    outs = []
    for shuffle in (True, True, False):
        w = synth.get("p_qwen_small").with_(shuffle_blocks=shuffle)
        s = WL.make_drafter(w, 2)
        WL.reset_sequences(s)
        out = WL.alloc_outputs(s)
        got = []
        for it in range(2):
            inp = WL.iter_inputs(s, it)
            WL.draft(s, it, inp, out)
            tl = WL.synthetic_target(s, it, out.logits)
            WL.verify(s, inp, tl, out)
            torch.cuda.synchronize()
            got.append((out.logits.cpu().numpy().copy(), out.drafts.cpu().numpy().copy(),
                        out.tokens.cpu().numpy().copy()))
        outs.append(got)
    for a, b in zip(outs[0], outs[1]):
        for x, y in zip(a, b):
            assert np.array_equal(x, y)
    for a, b in zip(outs[0], outs[2]):
        for x, y in zip(a, b):
            assert np.array_equal(x, y)


# ----------------------------------------------------------------------------------------
# full-size workloads, sampled sequences (the GPU runs the whole batch)
# ----------------------------------------------------------------------------------------
@pytest.mark.parametrize("name,seqs,iters", [("c2", [0], 2), ("c2t0", [0], 2), ("c2g", [0], 2),
                                             ("c3", [7], 2), ("c4", [30, 31], 2),
                                             ("c5", [62, 63], 2), ("osprey_2l", [0], 2),
                                             ("c2b", [0], 2), ("dflash_4l", [0], 2)])
def test_full_size_sampled_sequences_match_oracle(name, seqs, iters):
    """Benchmark-size shapes in the launch configuration the benchmark uses; the oracle
    follows the sampled sequences one by one (sequences of a batch are independent)."""
    _require_gpu()
    w = synth.get(name)
    stats = _run_parity(w, iters, seqs, 2e-2)
    assert stats["compared"] >= len(seqs)
    _assert_exact_comparisons(stats, name)


def test_block_with_packed_rows_matches_oracle():
    """Block drafting in explicit mode with packed taps (taps_stride 0) and several new
    tokens per sequence (3, 1, 2): the mask rows sit between the sequences' new rows,
    so the packed token and tap rows and the block rows are indexed apart."""
    _require_gpu()
    from oracle.block import draft_block
    from paper_2609_09338_amd import workload as WL
    w = synth.get("p_block")
    _say(f"[parity] {w.name}: packed explicit block")
    s = WL.make_drafter(w, 2)
    WL.reset_sequences(s)
    dr = OH.build_drafter(w)
    B, dev = w.batch, s.device
    n_new = [3, 1, 2][:B]
    rng = np.random.default_rng(31)
    toks = [rng.integers(0, w.vocab_target - 1, n) for n in n_new]
    taps = [synth.taps(w, 5, b, n) for b, n in enumerate(n_new)]
    u = synth.u_draft(w, 0)
    out = WL.alloc_outputs(s)
    s.drafter.draft_step(list(range(B)), w.K, WL.to_dev(np.concatenate(taps), w, dev),
                         s.draft_temperature, torch.from_numpy(u).to(dev), n_new=n_new,
                         new_tokens=torch.from_numpy(np.concatenate(toks).astype(np.int32)).to(dev),
                         taps_stride=0, draft_tokens=out.drafts, draft_logits=out.logits,
                         mask_token=synth.mask_token(w))
    torch.cuda.synchronize()
    assert s.drafter.device_errors() == 0
    g_logits, g_drafts = out.logits.cpu().numpy(), out.drafts.cpu().numpy()
    flagged = 0
    for b in range(B):
        seq = OH.start_sequence(w, dr, b, 2)
        Td = w.draft_temperature(b)
        drafts, logits, _, _ = draft_block(dr, seq, toks[b], taps[b].astype(np.float64), w.K, Td,
                                           u[b], synth.mask_token(w))
        for k in range(w.K):
            delta = _delta(g_logits[b, k], logits[k])
            assert delta <= 2e-2, (b, k, delta)
            if g_drafts[b, k] != drafts[k]:
                assert parity.draw_flag(logits[k], Td, float(u[b, k]), delta), (b, k)
                flagged += 1
    assert flagged <= 1


@pytest.mark.parametrize("name", ["p_single64", "p_partial"])
def test_draft_pick_extreme_uniforms(name):
    """Draws at u = 0, at and just below 1 and in between -- the inverse CDF's first
    entry, its rounding fallbacks at the end of the row, ordinary points -- pick what the oracle's
    inverse CDF picks on the same drafter logit rows (single sequences draw inside the
    next step's layer-0 projection, batches in the sampling kernel; p_partial leaves
    drafter rows unmapped)."""
    _require_gpu()
    from paper_2609_09338_amd import workload as WL
    w = synth.get(name)
    _say(f"[parity] {w.name}: draft picks at extreme uniforms")
    s = WL.make_drafter(w, 1)
    WL.reset_sequences(s)
    inp = WL.iter_inputs(s, 0)
    # (u = 1 lies outside the callers' [0, 1): it stands in for rounding that carries
    # u S past the total, where the pick takes the last entry with weight)
    pattern = [0.0, 1.0, 1.0 - 2.0 ** -24, 0.5, 2.0 ** -30, 0.999, 1.0 - 2.0 ** -20, 0.25]
    u = np.array([[pattern[(b + k) % len(pattern)] for k in range(w.K)] for b in range(w.batch)],
                 dtype=np.float32)
    inp.u_draft = torch.from_numpy(u).to(s.device)
    out = WL.alloc_outputs(s)
    WL.draft(s, 0, inp, out)
    torch.cuda.synchronize()
    assert s.drafter.device_errors() == 0
    g_logits, g_drafts = out.logits.cpu().numpy(), out.drafts.cpu().numpy()
    d2t = synth.make_d2t(w)
    exact = 0
    for b in range(w.batch):
        Td = w.draft_temperature(b)
        for k in range(w.K):
            row = g_logits[b, k].astype(np.float64)
            assert np.isfinite(row).any()
            mapped = set(int(t) for t in d2t[np.isfinite(row)])
            assert int(g_drafts[b, k]) in mapped, (b, k, g_drafts[b, k])
            want = int(d2t[OS.pick(row, Td, float(u[b, k]))])
            if int(g_drafts[b, k]) == want:
                exact += 1
            else:
                # the GPU's exponentials are fp32: allow a boundary within their error
                assert parity.draw_flag(row, Td, float(u[b, k]), 1e-5), (b, k, g_drafts[b, k], want)
    assert exact >= (w.batch * w.K) // 2, exact
