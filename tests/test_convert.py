"""The backbone-to-drafter conversion (paper_2609_09338_amd.convert) against what
Sections 3.2-3.3 fix.

* Eq. 2-3: the converted drafter computes exactly what the pruned backbone does,
  whatever the taps: the oracle drafter on the converted weights, fed random taps,
  matches transformers' Qwen3ForCausalLM with only the kept blocks, in float64
  (transformers computes RoPE angles in float32: ~1e-6).
* Pruning keeps the first blocks: changing a dropped block changes nothing.
* Vocabulary alignment: a shared token's row is copied, any other is the mean of
  the source rows of its text as the source tokenizer splits it (constructed
  vocabularies, exact), and the resized head is indexed by target id (d2t identity).
"""
import numpy as np
import pytest
import torch

import synth
from oracle.drafter import Drafter, Sequence
from paper_2609_09338_amd import convert

transformers = pytest.importorskip("transformers")


def _hf(n_layers, seed):
    from transformers import Qwen3Config, Qwen3ForCausalLM
    cfg = Qwen3Config(vocab_size=89, hidden_size=64, intermediate_size=96, num_hidden_layers=n_layers,
                      num_attention_heads=4, num_key_value_heads=2, head_dim=16, rms_norm_eps=1e-6,
                      max_position_embeddings=512,
                      rope_parameters={"rope_type": "default", "rope_theta": 1e6},
                      tie_word_embeddings=False)
    cfg._attn_implementation = "eager"
    torch.manual_seed(seed)
    m = Qwen3ForCausalLM(cfg).double().eval()
    g = torch.Generator().manual_seed(seed + 1)
    with torch.no_grad():   # norm gains away from 1, so that each one is exercised
        for name, p in m.named_parameters():
            if name.endswith("norm.weight"):
                p.copy_(1.0 + 0.1 * torch.randn(p.shape, generator=g, dtype=torch.float64))
    return m


def _state(m):
    return {k: v.detach().numpy().copy() for k, v in m.state_dict().items()}


def _workload(n_layers, vocab):
    return synth.Workload(name="conv", cfg_id=141, dtype="f32", n_layers=n_layers, d_model=64,
                          n_q_heads=4, n_kv_heads=2, head_dim=16, d_ffn=96, vocab_draft=vocab,
                          vocab_target=vocab, target_hidden=24, batch=1, K=3, prefill="ingest")


def _drafter_logits(w, weights, tokens, taps):
    dr = Drafter(w, weights, weights["d2t"])
    seq = Sequence(w, 64)
    s = dr.project_taps(taps)
    out = []
    for j, t in enumerate(tokens):
        g = dr.forward_row(seq, int(t), s[j], j)
        out.append(dr.logits(g))
    return np.array(out)


def test_converted_drafter_is_the_pruned_backbone_for_any_taps():
    full = _hf(3, 5)
    weights = convert.convert_qwen3(_state(full), 2, 3 * 24, rng=np.random.default_rng(3))
    pruned = _hf(2, 9)
    keep = {k: v for k, v in full.state_dict().items() if not k.startswith("model.layers.2.")}
    pruned.load_state_dict(keep, strict=True)
    rng = np.random.default_rng(11)
    tokens = rng.integers(0, 89, 9)
    with torch.no_grad():
        ref = pruned(torch.tensor(tokens[None])).logits[0].numpy()
    w = _workload(2, 89)
    for scale in (1.0, 30.0):
        got = _drafter_logits(w, weights, tokens, rng.standard_normal((9, 72)) * scale)
        assert np.max(np.abs(got - ref)) < 2e-6
    assert np.all(weights["layers.0.w_qkv"][:, :64] == 0.0)
    s = _state(full)
    np.testing.assert_array_equal(
        weights["layers.1.w_qkv"][:, 64:],
        np.concatenate([s["model.layers.1.self_attn." + n + "_proj.weight"] for n in "qkv"]))


def test_pruning_ignores_the_dropped_blocks():
    a, b = _hf(3, 5), _hf(3, 5)
    with torch.no_grad():
        for p in b.model.layers[2].parameters():
            p.add_(1.0)
    ca = convert.convert_qwen3(_state(a), 2, 72, rng=np.random.default_rng(0))
    cb = convert.convert_qwen3(_state(b), 2, 72, rng=np.random.default_rng(0))
    assert sorted(ca) == sorted(cb)
    for k in ca:
        np.testing.assert_array_equal(ca[k], cb[k])


def _greedy_tokenizer(vocab):
    """Longest match first over the vocabulary's strings; unknown characters are skipped."""
    def tok(text):
        ids, i = [], 0
        while i < len(text):
            for j in range(len(text), i, -1):
                if text[i:j] in vocab:
                    ids.append(vocab[text[i:j]])
                    i = j
                    break
            else:
                i += 1
        return ids
    return tok


def test_vocabulary_alignment_copies_shared_rows_and_averages_the_rest():
    src = {"a": 0, "b": 1, "c": 2, "ab": 3, "<s>": 4}
    tgt = {"ab": 0, "abc": 1, "ca": 2, "zz": 3, "b": 4}
    w = np.random.default_rng(2).standard_normal((5, 6))
    out = convert.align_rows(w, src, tgt, _greedy_tokenizer(src))
    np.testing.assert_array_equal(out[0], w[3])
    np.testing.assert_array_equal(out[1], (w[3] + w[2]) / 2)
    np.testing.assert_array_equal(out[2], (w[2] + w[0]) / 2)
    np.testing.assert_array_equal(out[3], np.zeros(6))
    np.testing.assert_array_equal(out[4], w[1])
    # a target text that differs from its token string (tgt_text)
    out2 = convert.align_rows(w, src, {"X": 0}, _greedy_tokenizer(src), tgt_text=lambda v: "cab")
    np.testing.assert_array_equal(out2[0], (w[2] + w[3]) / 2)


def test_converted_head_is_indexed_by_target_id():
    m = _hf(2, 7)
    src = {f"t{i}": i for i in range(89)}
    # the target keeps 40 source tokens under new ids and adds 9 made of two source tokens
    tgt = {f"t{i}": 48 - i for i in range(40)}
    tgt.update({f"t{i}t{i + 1}": 49 + i for i in range(9)})

    def tok(text):
        return [src["t" + p] for p in text.split("t")[1:]]
    c = convert.convert_qwen3(_state(m), 2, 72, vocab=dict(src_vocab=src, tgt_vocab=tgt, src_tokenize=tok))
    head = m.lm_head.weight.detach().numpy()
    emb = m.model.embed_tokens.weight.detach().numpy()
    assert c["lm_head"].shape == (58, 64) and c["embed"].shape == (58, 64)
    np.testing.assert_array_equal(c["d2t"], np.arange(58, dtype=np.int32))
    for i in range(40):
        np.testing.assert_array_equal(c["lm_head"][48 - i], head[i])
        np.testing.assert_array_equal(c["embed"][48 - i], emb[i])
    for i in range(9):
        np.testing.assert_array_equal(c["lm_head"][49 + i], (head[i] + head[i + 1]) / 2)
    # ids 0..8 are not used by this target vocabulary: zero rows
    assert np.all(c["lm_head"][:9] == 0.0)
