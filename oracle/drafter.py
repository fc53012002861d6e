"""The converted Osprey drafter, token by token, in float64.

Section 3.2 (Stage 1): the drafter keeps the embedding, the first N blocks,
the final norm and the LM head of a pretrained source LM.
Section 3.3: target hidden states from three layers are concatenated and
projected, c_t = W_c [h_low; h_mid; h_high] (Eq. 1); every attention layer's
QKV projection is widened to W~_qkv = [W^c  W_qkv] and applied to [c_{t-1}; z_t]
(Eq. 2-3), so the conditioning input s enters Q, K and V of every layer and
nothing else; vocabulary alignment gives an embedding indexed by target ids
and an LM head whose rows map to target ids through d2t (-1 = no target id).
Section 3.4: at draft steps the drafter's own hidden state takes the place of
the projected target state.

Readings where the paper is silent: no biases; s is used as is (no extra
norm); the position-0 input is zero; the fed-back state is the last layer's
residual output before the final norm; the body is the Qwen3 block (pre-norm
RMSNorm, per-head RMSNorm on q and k, rotate-half RoPE at absolute positions,
grouped-query attention, SwiGLU); cached keys and values are stored rounded to
bf16 in bf16 workloads.
"""
from __future__ import annotations

from typing import Dict, List, Tuple

import numpy as np

from . import numerics as nm
from . import sampling


def expected_shapes(cfg) -> Dict[str, Tuple[int, ...]]:
    """Shapes of every drafter tensor (what the conversion of Section 3.3 yields)."""
    d, hd = cfg.d_model, cfg.head_dim
    qkv = (cfg.n_q_heads + 2 * cfg.n_kv_heads) * hd
    s = {"embed": (cfg.vocab_target, d),                       # resized to |V_T| (Eq. 4)
         "w_c": (d, cfg.n_taps * cfg.target_hidden),            # Eq. 1
         "final_norm": (d,),
         "lm_head": (cfg.vocab_draft, d)}
    for l in range(cfg.n_layers):
        p = f"layers.{l}."
        s.update({p + "in_norm": (d,), p + "w_qkv": (qkv, 2 * d),   # Eq. 2: [W^c | W_qkv]
                  p + "q_norm": (hd,), p + "k_norm": (hd,), p + "w_o": (d, cfg.n_q_heads * hd),
                  p + "post_norm": (d,), p + "w_gate": (cfg.d_ffn, d), p + "w_up": (cfg.d_ffn, d),
                  p + "w_down": (d, cfg.d_ffn)})
    return s


def body_param_count(cfg) -> int:
    """Parameters of the transformer layers plus the hidden combiner W_c, i.e.
    what the paper's table of draft sizes counts (embedding and LM head excluded)."""
    shapes = expected_shapes(cfg)
    n = 0
    for name, shp in shapes.items():
        if name in ("embed", "lm_head", "final_norm"):
            continue
        if not cfg.qk_norm and (name.endswith("q_norm") or name.endswith("k_norm")):
            continue
        n += int(np.prod(shp))
    return n


class Sequence:
    """One sequence's drafter KV cache: [n_layers, capacity, n_kv, hd] keys and values."""

    def __init__(self, cfg, capacity: int):
        shp = (cfg.n_layers, capacity, cfg.n_kv_heads, cfg.head_dim)
        self.k = np.zeros(shp, dtype=np.float64)
        self.v = np.zeros(shp, dtype=np.float64)
        self.length = 0


class Drafter:
    def __init__(self, cfg, weights: Dict[str, np.ndarray], d2t: np.ndarray):
        self.cfg = cfg
        shapes = expected_shapes(cfg)
        self.w = {}
        for name, shp in shapes.items():
            a = np.asarray(weights[name], dtype=np.float64)
            if a.shape != shp:
                raise ValueError(f"{name}: shape {a.shape}, expected {shp}")
            self.w[name] = a
        self.d2t = np.asarray(d2t, dtype=np.int64)
        if self.d2t.shape != (cfg.vocab_draft,):
            raise ValueError("d2t must have one entry per LM-head row")
        self.kv_bf16 = cfg.dtype == "bf16"

    # -- Eq. 1 ---------------------------------------------------------------
    def project_taps(self, taps: np.ndarray) -> np.ndarray:
        """c = W_c [h_low; h_mid; h_high] for each row of taps [rows, n_taps * H]."""
        return np.asarray(taps, dtype=np.float64) @ self.w["w_c"].T

    # -- one position through the body ----------------------------------------
    def forward_row(self, seq: Sequence, token: int, s: np.ndarray, pos: int) -> np.ndarray:
        """Run target-id `token` at absolute position `pos` with conditioning
        input s; appends its keys/values to the cache; returns the last
        layer's residual output g (before the final norm)."""
        cfg, w = self.cfg, self.w
        d, hd, nq, nkv = cfg.d_model, cfg.head_dim, cfg.n_q_heads, cfg.n_kv_heads
        x = w["embed"][int(token)].copy()
        s = np.asarray(s, dtype=np.float64)
        for l in range(cfg.n_layers):
            p = f"layers.{l}."
            z = nm.rmsnorm(x, w[p + "in_norm"], cfg.rms_eps)
            qkv = w[p + "w_qkv"] @ np.concatenate([s, z])           # Eq. 2-3
            q = qkv[: nq * hd].reshape(nq, hd)
            k = qkv[nq * hd: (nq + nkv) * hd].reshape(nkv, hd)
            v = qkv[(nq + nkv) * hd:].reshape(nkv, hd)
            if cfg.qk_norm:
                q = nm.rmsnorm(q, w[p + "q_norm"], cfg.rms_eps)
                k = nm.rmsnorm(k, w[p + "k_norm"], cfg.rms_eps)
            q = nm.rope_rotate_half(q, pos, cfg.rope_theta)
            k = nm.rope_rotate_half(k, pos, cfg.rope_theta)
            if self.kv_bf16:
                k, v = nm.bf16_rne(k), nm.bf16_rne(v)
            seq.k[l, pos] = k
            seq.v[l, pos] = v
            o = nm.attention(q, seq.k[l, : pos + 1], seq.v[l, : pos + 1])
            x = x + w[p + "w_o"] @ o.reshape(-1)
            y = nm.rmsnorm(x, w[p + "post_norm"], cfg.rms_eps)
            x = x + w[p + "w_down"] @ (nm.silu(w[p + "w_gate"] @ y) * (w[p + "w_up"] @ y))
        seq.length = max(seq.length, pos + 1)
        return x

    def logits(self, g: np.ndarray) -> np.ndarray:
        """LM-head logits over drafter rows; rows with no target id are -inf."""
        h = nm.rmsnorm(g, self.w["final_norm"], self.cfg.rms_eps)
        l = self.w["lm_head"] @ h
        l[self.d2t < 0] = -np.inf
        return l

    # -- one draft call ---------------------------------------------------------
    def ingest(self, seq: Sequence, tokens, taps) -> np.ndarray:
        """Append committed tokens (target ids) whose conditioning rows are the
        projected taps of the preceding positions.  Returns the last row's g."""
        s_rows = self.project_taps(taps)
        g = None
        for tok, s in zip(tokens, s_rows):
            g = self.forward_row(seq, int(tok), s, seq.length)
        return g

    def draft(self, seq: Sequence, tokens, taps, K: int, T: float, u_draft):
        """Ingest the newly committed tokens, then propose K drafts.

        Returns (drafts [K] target ids, logits [K, V_d], draft_rows [K],
        committed_length).  Draft k is sampled from the logits of step k with
        uniform u_draft[k]; step k >= 1 feeds draft k-1 with the previous
        step's hidden state as its conditioning input."""
        g = self.ingest(seq, tokens, taps)
        committed = seq.length
        drafts, rows, logit_rows = [], [], []
        for k in range(K):
            if k > 0:
                g = self.forward_row(seq, drafts[-1], g, committed + k - 1)
            l = self.logits(g)
            r = sampling.pick(l, T, float(u_draft[k]))
            rows.append(r)
            drafts.append(int(self.d2t[r]))
            logit_rows.append(l)
        L = np.stack(logit_rows) if K else np.zeros((0, self.cfg.vocab_draft))
        return np.array(drafts, dtype=np.int64), L, np.array(rows, dtype=np.int64), committed

    def rollback(self, seq: Sequence, length: int) -> None:
        """Discard cached positions at or beyond `length` (the draft positions)."""
        seq.length = length
