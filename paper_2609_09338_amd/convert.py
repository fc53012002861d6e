"""Conversion of a pretrained next-token backbone into a drafter (Stages 1 and 3 of
Section 3), host-side, in the weight layout `osprey_weights` takes.

* Pruning (Stage 1, Section 3.2): keep the embedding, the LM head, the final norm and
  the first `n_layers` transformer blocks.
* Tap projection (Eq. 1): W_c [d, n_taps H] is new.  Its initial values do not
  matter at conversion (they multiply zero columns); they are drawn N(0, std).
* Zero-initialised QKV expansion (Eq. 2-3): each block's query, key and value
  projections are stacked into W_qkv and widened to [0  W_qkv], the zero columns
  taking the conditioning input c_{t-1}; at conversion W~ [c; z] = W_qkv z, so the
  drafter computes exactly what the pruned backbone did.  The library's column order
  is the same: columns [0, d) for c, [d, 2d) for the token-side input z.
* Vocabulary alignment (Section 3.3, last equation): the embedding and LM head are
  resized to the target vocabulary.  A target token that the source vocabulary holds
  keeps its source row; any other is the mean of the source rows of its text as the
  source tokenizer splits it.  The drafter then predicts target ids directly: d2t is
  the identity.

Reading where the paper is silent: a target token whose text the source tokenizer
maps to no token at all gets a zero row.

All arrays are numpy; the caller rounds them to the storage dtype and copies them to
the device (see `binding.Drafter`)."""
from __future__ import annotations

from typing import Callable, Dict, Mapping, Optional, Sequence

import numpy as np


def expand_qkv(w_q: np.ndarray, w_k: np.ndarray, w_v: np.ndarray) -> np.ndarray:
    """[0  W_qkv] with W_qkv = [W_q; W_k; W_v] (Eq. 2): shape [(n_q + 2 n_kv) hd, 2 d],
    zero in the first d columns (the conditioning input's)."""
    w = np.concatenate([np.asarray(w_q), np.asarray(w_k), np.asarray(w_v)], axis=0)
    return np.concatenate([np.zeros_like(w), w], axis=1)


def align_rows(w_src: np.ndarray, src_vocab: Mapping[str, int], tgt_vocab: Mapping[str, int],
               src_tokenize: Callable[[str], Sequence[int]],
               tgt_text: Optional[Callable[[str], str]] = None) -> np.ndarray:
    """Resize a source embedding or LM-head matrix to the target vocabulary.

    src_vocab / tgt_vocab map token strings to ids; target row tgt_vocab[v] is
    w_src[src_vocab[v]] when v is a source token, else the mean of w_src over
    src_tokenize(tgt_text(v)) (tgt_text defaults to the token string itself), or
    zero when that is empty."""
    w_src = np.asarray(w_src)
    n_t = max(tgt_vocab.values()) + 1 if tgt_vocab else 0
    out = np.zeros((n_t, w_src.shape[1]), dtype=w_src.dtype)
    text = tgt_text or (lambda v: v)
    for v, j in tgt_vocab.items():
        i = src_vocab.get(v)
        if i is not None:
            out[j] = w_src[i]
            continue
        ids = list(src_tokenize(text(v)))
        if ids:
            out[j] = np.mean(w_src[np.asarray(ids, dtype=np.int64)], axis=0)
    return out


def convert_qwen3(state: Mapping[str, np.ndarray], n_layers: int, tap_width: int,
                  rng: Optional[np.random.Generator] = None, w_c_std: float = 0.02,
                  vocab: Optional[dict] = None) -> Dict[str, np.ndarray]:
    """A Qwen3-style state dict (transformers naming: model.embed_tokens.weight,
    model.layers.{i}.self_attn.{q,k,v,o}_proj.weight, ...q_norm / k_norm,
    input_layernorm, post_attention_layernorm, mlp.{gate,up,down}_proj, model.norm,
    lm_head.weight, or tied embeddings) to the library's weights, keeping the first
    n_layers blocks.

    vocab, when given, holds src_vocab, tgt_vocab and src_tokenize (optionally
    tgt_text) for align_rows; without it the target shares the source vocabulary.
    Returns the weights by the library's names plus "d2t" (int32 identity)."""
    g = rng if rng is not None else np.random.default_rng(0)
    f = lambda k: np.asarray(state[k])
    embed = f("model.embed_tokens.weight")
    head = f("lm_head.weight") if "lm_head.weight" in state else embed
    if vocab is not None:
        kw = dict(src_vocab=vocab["src_vocab"], tgt_vocab=vocab["tgt_vocab"],
                  src_tokenize=vocab["src_tokenize"], tgt_text=vocab.get("tgt_text"))
        embed = align_rows(embed, **kw)
        head = align_rows(head, **kw)
    d = embed.shape[1]
    out = {"embed": embed, "lm_head": head, "final_norm": f("model.norm.weight"),
           "w_c": (g.standard_normal((d, tap_width)) * w_c_std).astype(embed.dtype)}
    for l in range(n_layers):
        s = f"model.layers.{l}."
        p = f"layers.{l}."
        out[p + "in_norm"] = f(s + "input_layernorm.weight")
        out[p + "w_qkv"] = expand_qkv(f(s + "self_attn.q_proj.weight"), f(s + "self_attn.k_proj.weight"),
                                      f(s + "self_attn.v_proj.weight"))
        out[p + "q_norm"] = f(s + "self_attn.q_norm.weight")
        out[p + "k_norm"] = f(s + "self_attn.k_norm.weight")
        out[p + "w_o"] = f(s + "self_attn.o_proj.weight")
        out[p + "post_norm"] = f(s + "post_attention_layernorm.weight")
        out[p + "w_gate"] = f(s + "mlp.gate_proj.weight")
        out[p + "w_up"] = f(s + "mlp.up_proj.weight")
        out[p + "w_down"] = f(s + "mlp.down_proj.weight")
    out["d2t"] = np.arange(head.shape[0], dtype=np.int32)
    return out
