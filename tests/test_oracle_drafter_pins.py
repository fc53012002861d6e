"""Pins of the oracle drafter against things other than itself.

* Eq. 3 (zero-initialised expansion): with the c-slot columns of W~_qkv zero,
  the drafter's logits do not depend on the target taps at all (bitwise), and
  equal those of an independent library decoder, transformers' Qwen3 model,
  run in float64 on the same weights (the pruned source LM of Section 3.2 is a
  Qwen3 model).  transformers computes RoPE angles in float32, which bounds the
  agreement at ~1e-6.
* Eq. 2 (expanded QKV on [c; z]): with the same conditioning input s at every
  position, W^c s is a constant added to q, k and v, i.e. exactly a Qwen3
  model with Q/K/V biases equal to the three slices of W^c s.
* RoPE is a rotation whose score depends on relative position only; attention
  over one position returns its value; identical keys average the values.
* bf16 cache rounding equals torch's float -> bfloat16 conversion.
* Shapes: the parameter counts implied by the converted drafter's tensors
  reproduce the paper's table of draft sizes (Appendix E).
"""
import numpy as np
import pytest
import torch

import synth
from oracle import numerics as nm
from oracle.drafter import Drafter, Sequence, body_param_count

transformers = pytest.importorskip("transformers")


def _tiny(**kw):
    base = dict(name="pin", cfg_id=101, dtype="f32", n_layers=2, d_model=64, n_q_heads=4,
                n_kv_heads=2, head_dim=16, d_ffn=96, vocab_draft=97, vocab_target=97,
                target_hidden=24, batch=1, K=3, prefill="ingest", gains="normal")
    base.update(kw)
    return synth.Workload(**base)


def _hf_model(w, weights, bias_s=None):
    from transformers import Qwen3Config, Qwen3ForCausalLM
    cfg = Qwen3Config(vocab_size=w.vocab_target, hidden_size=w.d_model,
                      intermediate_size=w.d_ffn, num_hidden_layers=w.n_layers,
                      num_attention_heads=w.n_q_heads, num_key_value_heads=w.n_kv_heads,
                      head_dim=w.head_dim, rms_norm_eps=w.rms_eps, max_position_embeddings=4096,
                      rope_parameters={"rope_type": "default", "rope_theta": w.rope_theta},
                      tie_word_embeddings=False, attention_bias=bias_s is not None)
    cfg._attn_implementation = "eager"
    torch.manual_seed(0)
    m = Qwen3ForCausalLM(cfg).double().eval()
    d, hd, nq, nkv = w.d_model, w.head_dim, w.n_q_heads, w.n_kv_heads
    t = lambda a: torch.tensor(np.asarray(a, dtype=np.float64))
    with torch.no_grad():
        m.model.embed_tokens.weight.copy_(t(weights["embed"]))
        m.model.norm.weight.copy_(t(weights["final_norm"]))
        m.lm_head.weight.copy_(t(weights["lm_head"]))
        for l, layer in enumerate(m.model.layers):
            p = f"layers.{l}."
            wq = np.asarray(weights[p + "w_qkv"], dtype=np.float64)
            tok = wq[:, d:]
            a = layer.self_attn
            a.q_proj.weight.copy_(t(tok[: nq * hd]))
            a.k_proj.weight.copy_(t(tok[nq * hd:(nq + nkv) * hd]))
            a.v_proj.weight.copy_(t(tok[(nq + nkv) * hd:]))
            if bias_s is not None:
                b = wq[:, :d] @ bias_s
                a.q_proj.bias.copy_(t(b[: nq * hd]))
                a.k_proj.bias.copy_(t(b[nq * hd:(nq + nkv) * hd]))
                a.v_proj.bias.copy_(t(b[(nq + nkv) * hd:]))
            a.q_norm.weight.copy_(t(weights[p + "q_norm"]))
            a.k_norm.weight.copy_(t(weights[p + "k_norm"]))
            a.o_proj.weight.copy_(t(weights[p + "w_o"]))
            layer.input_layernorm.weight.copy_(t(weights[p + "in_norm"]))
            layer.post_attention_layernorm.weight.copy_(t(weights[p + "post_norm"]))
            layer.mlp.gate_proj.weight.copy_(t(weights[p + "w_gate"]))
            layer.mlp.up_proj.weight.copy_(t(weights[p + "w_up"]))
            layer.mlp.down_proj.weight.copy_(t(weights[p + "w_down"]))
    return m


def _oracle_logits_per_position(w, weights, tokens, taps):
    dr = Drafter(w, weights, np.arange(w.vocab_draft))
    seq = Sequence(w, len(tokens) + 1)
    s_rows = dr.project_taps(taps)
    out = []
    for tok, s in zip(tokens, s_rows):
        g = dr.forward_row(seq, int(tok), s, seq.length)
        out.append(dr.logits(g))
    return np.stack(out)


def _hf_logits(m, tokens):
    with torch.no_grad():
        ids = torch.tensor(np.asarray(tokens, dtype=np.int64))[None]
        return m(input_ids=ids).logits[0].numpy()


def test_zero_expansion_is_independent_of_taps_bitwise():
    w = _tiny(expansion="zero")
    weights = synth.make_weights(w)
    toks = synth.prompt_tokens(w, 0, 11)
    rng = np.random.default_rng(5)
    a = _oracle_logits_per_position(w, weights, toks, rng.standard_normal((11, w.tap_width)))
    b = _oracle_logits_per_position(w, weights, toks, np.zeros((11, w.tap_width)))
    assert np.array_equal(a, b)


def test_zero_expansion_equals_library_qwen3_decoder():
    w = _tiny(expansion="zero")
    weights = synth.make_weights(w)
    toks = synth.prompt_tokens(w, 0, 23)
    taps = np.random.default_rng(6).standard_normal((23, w.tap_width))
    ours = _oracle_logits_per_position(w, weights, toks, taps)
    ref = _hf_logits(_hf_model(w, weights), toks)
    assert np.max(np.abs(ref)) > 0.1
    np.testing.assert_allclose(ours, ref, atol=2e-6, rtol=0)


def test_constant_conditioning_equals_qwen3_with_qkv_bias():
    w = _tiny(expansion="normal", d_model=64, n_q_heads=8, n_kv_heads=2, head_dim=8)
    weights = synth.make_weights(w)
    toks = synth.prompt_tokens(w, 1, 17)
    tap = np.random.default_rng(7).standard_normal(w.tap_width)
    taps = np.tile(tap, (17, 1))
    ours = _oracle_logits_per_position(w, weights, toks, taps)
    s = np.asarray(weights["w_c"], dtype=np.float64) @ tap
    ref = _hf_logits(_hf_model(w, weights, bias_s=s), toks)
    # the bias actually changes the function (so the test has power) ...
    plain = _hf_logits(_hf_model(w, weights), toks)
    assert np.max(np.abs(plain - ref)) > 1e-2
    # ... and the oracle matches it
    np.testing.assert_allclose(ours, ref, atol=2e-6, rtol=0)


def test_rope_scores_depend_on_relative_position_only():
    rng = np.random.default_rng(8)
    q, k = rng.standard_normal(64), rng.standard_normal(64)
    base = nm.rope_rotate_half(q, 37, 1e6) @ nm.rope_rotate_half(k, 5, 1e6)
    for shift in (1, 100, 4000):
        s = nm.rope_rotate_half(q, 37 + shift, 1e6) @ nm.rope_rotate_half(k, 5 + shift, 1e6)
        assert abs(s - base) < 1e-9
    # a rotation: norms preserved, position 0 is the identity
    assert abs(np.linalg.norm(nm.rope_rotate_half(q, 1234, 1e4)) - np.linalg.norm(q)) < 1e-12
    np.testing.assert_array_equal(nm.rope_rotate_half(q, 0, 1e6), q)


def test_attention_special_cases():
    rng = np.random.default_rng(9)
    q = rng.standard_normal((4, 16))
    k1, v1 = rng.standard_normal((1, 2, 16)), rng.standard_normal((1, 2, 16))
    o = nm.attention(q, k1, v1)
    np.testing.assert_allclose(o[:2], np.broadcast_to(v1[0, 0], (2, 16)), atol=1e-15)
    np.testing.assert_allclose(o[2:], np.broadcast_to(v1[0, 1], (2, 16)), atol=1e-15)
    k = np.broadcast_to(rng.standard_normal((1, 2, 16)), (9, 2, 16))
    v = rng.standard_normal((9, 2, 16))
    o = nm.attention(q, k, v)
    np.testing.assert_allclose(o[0], v[:, 0].mean(0), atol=1e-13)
    np.testing.assert_allclose(o[3], v[:, 1].mean(0), atol=1e-13)


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(10)
    x = (rng.standard_normal(200000) * np.exp(rng.uniform(-20, 20, 200000))).astype(np.float32)
    x[:4] = [1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -(1.0 + 2 ** -8), 0.0]   # exact ties
    ours = nm.bf16_rne(x.astype(np.float64))
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(ours, ref)


def _printed_sizes():
    import os
    path = os.path.join(os.path.dirname(__file__), "golden", "draft_sizes.txt")
    out = {}
    for line in open(path):
        line = line.split("#")[0].split()
        if line:
            out[line[0]] = (float(line[1]) * 1e6, float(line[2]) * 1e6)
    return out


# Osprey: two blocks of Qwen3-4B (d 2560, 32/8 heads, head_dim 128, FFN 9728, QK-norm);
# LayerSkip: four blocks of Llama-3.2-1B (d 2048, 32/8 heads, head_dim 64, FFN 8192).
_OSPREY = dict(n_layers=2, d_model=2560, n_q_heads=32, n_kv_heads=8, head_dim=128, d_ffn=9728,
               qk_norm=1)
_LAYERSKIP = dict(n_layers=4, d_model=2048, n_q_heads=32, n_kv_heads=8, head_dim=64,
                  d_ffn=8192, qk_norm=0)


@pytest.mark.parametrize("key,kw", [("osprey_2l_body", _OSPREY),
                                    ("layerskip_4l_body", _LAYERSKIP)])
def test_body_parameter_counts_match_paper_table(key, kw):
    # conditioned on Qwen3-8B: three taps of its 4096-wide hidden state
    printed, rounding = _printed_sizes()[key]
    n = body_param_count(_tiny(target_hidden=4096, **kw))
    assert abs(n - printed) <= rounding / 2, (key, n)


@pytest.mark.parametrize("key,kw,vocab", [("qwen3_4b_2l_pruned", _OSPREY, 151936),
                                          ("layerskip_4l_pruned", _LAYERSKIP, 128256)])
def test_pruned_backbone_sizes(key, kw, vocab):
    # before conversion: no W_c, no c-slot columns, one (tied) vocab x d table and the final norm
    printed, rounding = _printed_sizes()[key]
    w = _tiny(target_hidden=4096, vocab_draft=vocab, vocab_target=vocab, **kw)
    c_cols = w.n_layers * w.qkv_rows * w.d_model
    n = body_param_count(w) - c_cols - w.d_model * w.tap_width + vocab * w.d_model + w.d_model
    assert abs(n - printed) <= rounding / 2, (key, n)


def _hf_model_mapped(w, weights, d2t):
    """transformers' Qwen3 over target ids: its output layer holds, for every target id,
    the LM-head row that maps to it (zero when none does; those ids are masked below)."""
    lm = np.zeros((w.vocab_target, w.d_model))
    rows = np.flatnonzero(d2t >= 0)
    lm[d2t[rows]] = np.asarray(weights["lm_head"], dtype=np.float64)[rows]
    return _hf_model(w, dict(weights, lm_head=lm))


@pytest.mark.parametrize("vmap,V_d", [("identity", 97), ("inject", 61)])
def test_greedy_chain_equals_library_qwen3_greedy_continuation(vmap, V_d):
    """Section 3.4's autoregressive loop (step k >= 1 feeds draft k-1 at position
    committed + k - 1).  With the expansion columns zero (Eq. 3) the fed-back hidden
    state is multiplied by zero, so the drafter is its pruned backbone and a T = 0
    chain of K drafts must be transformers' Qwen3 greedy continuation of the committed
    prefix: the same fed tokens at the same positions, logits within the float32-RoPE
    tolerance, drafts emitted as target ids through the vocabulary map.  The prefix
    arrives in two draft calls, the first one's drafts rolled back, so the committed
    length carried between calls is pinned as well."""
    w = _tiny(expansion="zero", vocab_draft=V_d, vocab_map=vmap, K=5)
    weights = synth.make_weights(w)
    d2t = synth.make_d2t(w)
    dr = Drafter(w, weights, d2t)
    prefix = synth.prompt_tokens(w, 2, 13)
    taps = np.random.default_rng(12).standard_normal((13, w.tap_width))
    seq = Sequence(w, 32)
    _, _, _, committed = dr.draft(seq, prefix[:9], taps[:9], 2, 0.0, np.zeros(2))
    assert committed == 9
    dr.rollback(seq, committed)
    drafts, logits, rows, committed = dr.draft(seq, prefix[9:], taps[9:], w.K, 0.0, np.zeros(w.K))
    assert committed == 13
    m = _hf_model_mapped(w, weights, d2t)
    reach = np.zeros(w.vocab_target, dtype=bool)
    reach[d2t[d2t >= 0]] = True
    ids = [int(t) for t in prefix]
    for k in range(w.K):
        ref = _hf_logits(m, ids)[-1]
        ref[~reach] = -np.inf
        ours = np.full(w.vocab_target, -np.inf)
        mapped = d2t >= 0
        ours[d2t[mapped]] = logits[k][mapped]
        assert np.array_equal(np.isfinite(ours), np.isfinite(ref))
        fin = np.isfinite(ref)
        np.testing.assert_allclose(ours[fin], ref[fin], atol=2e-6, rtol=0)
        top2 = np.sort(ref[fin])[-2:]
        assert top2[1] - top2[0] > 1e-4          # no near tie: the argmax is decided
        nxt = int(np.argmax(ref))
        assert int(drafts[k]) == nxt, (k, int(drafts[k]), nxt)
        assert int(d2t[rows[k]]) == nxt
        ids.append(nxt)
