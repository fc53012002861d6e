"""Seeded synthetic inputs for the Osprey draft-and-verify step.

This module is the only code shared by the GPU path's tests and benchmark and
by the CPU oracle.  It holds no arithmetic of the method: it draws random
numbers, rounds generated values to the bf16 storage grid (a property of the
inputs, not of the method), and describes the workloads.  Every random stream
is `numpy.random.default_rng(SeedSequence((workload id, variant, stream, ...)))`
so that any consumer can regenerate any piece independently.

Workloads stand in for the paper's serving settings (Section 4 "Inference
settings", Appendix D.1 serving sensitivity): the paper's trained weights,
target models and evaluation prompts are not available, so weights are
N(0, 0.02), target hidden states are N(0, 1), token ids are uniform, and the
target's logits are the drafter's logits plus Gaussian noise (see
`target_logits`).
"""
from __future__ import annotations

import dataclasses
from dataclasses import dataclass, field
from typing import Dict, List, Tuple

import numpy as np

# Stream ids (third SeedSequence key).
S_WEIGHTS, S_VOCAB, S_PROMPT, S_TAPS, S_CTX_KV, S_NOISE, S_U_DRAFT, S_U_ACC, \
    S_U_BONUS, S_CTX_LEN, S_BLOCKS = range(11)


@dataclass(frozen=True)
class Workload:
    name: str
    cfg_id: int
    dtype: str                 # "f32" or "bf16": weights, taps and KV storage
    n_layers: int
    d_model: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    d_ffn: int
    vocab_draft: int           # LM-head rows
    vocab_target: int          # embedding rows and verify width
    target_hidden: int         # width of one target hidden-state tap
    n_taps: int = 3
    qk_norm: int = 1
    rms_eps: float = 1e-6
    rope_theta: float = 1.0e6
    batch: int = 1
    K: int = 4
    ctx_lo: int = 128          # committed length before the first draft
    ctx_hi: int = 128          # contexts ~ U[ctx_lo, ctx_hi] per sequence
    prefill: str = "kv"        # "kv": synthetic post-RoPE KV; "ingest": prompt run through the drafter
    temps: Tuple[float, ...] = (0.0,)   # temperature of request b is temps[b % len(temps)]
    draft_temps: Tuple[float, ...] = ()  # drafter's temperature per request (empty: = temps)
    sigma: float = 1.0         # std of the noise added to form target logits
    vocab_map: str = "identity"  # "identity" | "inject" | "partial"
    expansion: str = "normal"  # "zero" | "normal": the c-slot columns of W~_qkv
    gains: str = "one"         # "one" | "normal": RMSNorm gains 1 or 1 + N(0, 0.1)
    kv_block: int = 16
    shuffle_blocks: bool = False
    variant: int = 0
    drafting: str = "chain"    # "chain": K autoregressive steps; "block": one block pass

    def with_(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)

    @property
    def qkv_rows(self) -> int:
        return (self.n_q_heads + 2 * self.n_kv_heads) * self.head_dim

    @property
    def tap_width(self) -> int:
        return self.n_taps * self.target_hidden

    def temperature(self, b: int) -> float:
        return float(self.temps[b % len(self.temps)])

    def draft_temperature(self, b: int) -> float:
        """Temperature the drafter samples request b at (0: greedy drafting)."""
        if not self.draft_temps:
            return self.temperature(b)
        return float(self.draft_temps[b % len(self.draft_temps)])


def mask_token(w: "Workload") -> int:
    """The placeholder token of block drafting: the last target id."""
    return w.vocab_target - 1


# ---------------------------------------------------------------------------
# The five benchmark workloads and smaller parity shapes.
# ---------------------------------------------------------------------------
_QWEN_DRAFTER = dict(dtype="bf16", n_layers=2, d_model=1024, n_q_heads=16, n_kv_heads=8,
                     head_dim=128, d_ffn=3072)

WORKLOADS: Dict[str, Workload] = {
    # Tiny fp32 chain draft (1-layer, d 256, V_d 2048 injected into V_T 4096).
    "c1": Workload(name="c1", cfg_id=1, dtype="f32", n_layers=1, d_model=256, n_q_heads=4,
                   n_kv_heads=4, head_dim=64, d_ffn=1024, vocab_draft=2048, vocab_target=4096,
                   target_hidden=512, batch=1, K=4, ctx_lo=128, ctx_hi=128, prefill="ingest",
                   temps=(0.0,), sigma=0.5, vocab_map="inject", expansion="normal"),
    # Qwen3-8B-shaped target, batch 1, context 2048, K = 7.
    "c2": Workload(name="c2", cfg_id=2, vocab_draft=151936, vocab_target=151936,
                   target_hidden=4096, batch=1, K=7, ctx_lo=2048, ctx_hi=2048, temps=(1.0,),
                   sigma=1.0, **_QWEN_DRAFTER),
    # The same step with a greedy target (T = 0; the other temperature the configuration
    # names): prefix match against the target's argmax, bonus = argmax.
    "c2t0": Workload(name="c2t0", cfg_id=10, vocab_draft=151936, vocab_target=151936,
                     target_hidden=4096, batch=1, K=7, ctx_lo=2048, ctx_hi=2048, temps=(0.0,),
                     sigma=1.0, **_QWEN_DRAFTER),
    # Llama-3.3-70B-shaped target: partial surjective map 151936 -> 128256.
    "c3": Workload(name="c3", cfg_id=3, vocab_draft=151936, vocab_target=128256,
                   target_hidden=8192, batch=8, K=6, ctx_lo=4096, ctx_hi=4096, temps=(1.0,),
                   sigma=1.0, vocab_map="partial", **_QWEN_DRAFTER),
    # Large-vocab MoE-scale target: 151936 injected into 200064, paged shuffled KV.
    "c4": Workload(name="c4", cfg_id=4, vocab_draft=151936, vocab_target=200064,
                   target_hidden=3072, batch=32, K=5, ctx_lo=8192, ctx_hi=8192, temps=(0.7,),
                   sigma=1.5, vocab_map="inject", shuffle_blocks=True, **_QWEN_DRAFTER),
    # The Qwen3-8B-shaped step with greedy (top-1) drafting verified against a target
    # sampled at T = 1: the serving setup the paper reports (top-1 chains).
    "c2g": Workload(name="c2g", cfg_id=6, vocab_draft=151936, vocab_target=151936,
                    target_hidden=4096, batch=1, K=7, ctx_lo=2048, ctx_hi=2048, temps=(1.0,),
                    draft_temps=(0.0,), sigma=1.0, **_QWEN_DRAFTER),
    # The paper's own drafter shape (2 layers of pruned Qwen3-4B: d 2560, 32 / 8 heads x 128,
    # FFN 9728; its size is pinned by the table of draft sizes) for the Qwen3-8B target,
    # served as the paper serves it: a greedy (top-1) chain of 5 draft steps, target
    # temperature 0; a target close to the drafter (sigma 0.05) stands in for a trained one.
    "osprey_2l": Workload(name="osprey_2l", cfg_id=7, dtype="bf16", n_layers=2, d_model=2560,
                          n_q_heads=32, n_kv_heads=8, head_dim=128, d_ffn=9728,
                          vocab_draft=151936, vocab_target=151936, target_hidden=4096, batch=1,
                          K=5, ctx_lo=2048, ctx_hi=2048, temps=(0.0,), draft_temps=(0.0,),
                          sigma=0.05),
    # Throughput-bound decode: batch 64, ragged contexts, mixed greedy / T = 1.
    "c5": Workload(name="c5", cfg_id=5, vocab_draft=151936, vocab_target=151936,
                   target_hidden=4096, batch=64, K=7, ctx_lo=512, ctx_hi=4096,
                   temps=(0.0, 1.0), sigma=1.0, shuffle_blocks=True, **_QWEN_DRAFTER),
    # Block drafting (the EAGLE-style interface of the DFlash ablation) with the c2 drafter:
    # 7 proposals from one pass over the anchor and 6 mask rows.
    "c2b": Workload(name="c2b", cfg_id=8, vocab_draft=151936, vocab_target=151936,
                    target_hidden=4096, batch=1, K=7, ctx_lo=2048, ctx_hi=2048, temps=(1.0,),
                    sigma=1.0, drafting="block", **_QWEN_DRAFTER),
    # The ablation's own shape: a four-block Llama-shaped drafter (d 2048, 32 / 8 heads x
    # 64, FFN 8192, no QK-norm, RoPE theta 5e5) for the Qwen3-8B target, blocks of 16
    # (15 proposals).
    "dflash_4l": Workload(name="dflash_4l", cfg_id=9, dtype="bf16", n_layers=4, d_model=2048,
                          n_q_heads=32, n_kv_heads=8, head_dim=64, d_ffn=8192, qk_norm=0,
                          rope_theta=5.0e5, vocab_draft=151936, vocab_target=151936,
                          target_hidden=4096, batch=1, K=15, ctx_lo=2048, ctx_hi=2048,
                          temps=(1.0,), sigma=1.0, drafting="block"),
}

# Parity shapes: the benchmark architectures at sizes the oracle finishes in
# seconds, with ragged vocabularies (not multiples of any tile), contexts that
# straddle KV-block boundaries and several sequences per batch.
PARITY: Dict[str, Workload] = {
    "p_tiny_f32": WORKLOADS["c1"].with_(name="p_tiny_f32", cfg_id=11),
    "p_qwen_small": Workload(name="p_qwen_small", cfg_id=12, dtype="bf16", n_layers=2,
                             d_model=256, n_q_heads=4, n_kv_heads=2, head_dim=64, d_ffn=768,
                             vocab_draft=5003, vocab_target=5003, target_hidden=320, batch=3,
                             K=5, ctx_lo=17, ctx_hi=49, temps=(0.0, 1.0, 0.7), sigma=1.0,
                             shuffle_blocks=True),
    "p_partial": Workload(name="p_partial", cfg_id=13, dtype="bf16", n_layers=2, d_model=512,
                          n_q_heads=8, n_kv_heads=4, head_dim=64, d_ffn=1024, vocab_draft=6007,
                          vocab_target=4099, target_hidden=256, batch=4, K=6, ctx_lo=31,
                          ctx_hi=65, temps=(1.0,), sigma=1.0, vocab_map="partial",
                          shuffle_blocks=True),
    # greedy drafting against sampled, greedy and sharply sampled targets
    "p_greedy_draft": Workload(name="p_greedy_draft", cfg_id=15, dtype="bf16", n_layers=2,
                               d_model=256, n_q_heads=4, n_kv_heads=2, head_dim=64, d_ffn=768,
                               vocab_draft=5003, vocab_target=4099, target_hidden=320,
                               batch=4, K=5, ctx_lo=9, ctx_hi=40, temps=(1.0, 0.1, 0.0, 0.7),
                               draft_temps=(0.0, 0.0, 0.0, 0.3), sigma=0.05,
                               vocab_map="partial", shuffle_blocks=True),
    # single sequences (batch 1): the one-launch body of autoregressive steps
    "p_single64": Workload(name="p_single64", cfg_id=16, dtype="bf16", n_layers=2, d_model=256,
                           n_q_heads=8, n_kv_heads=2, head_dim=64, d_ffn=640, vocab_draft=4001,
                           vocab_target=4001, target_hidden=128, batch=1, K=6, ctx_lo=23,
                           ctx_hi=23, temps=(1.0,), sigma=0.5, shuffle_blocks=True),
    "p_single128": Workload(name="p_single128", cfg_id=17, dtype="bf16", n_layers=3, d_model=384,
                            n_q_heads=4, n_kv_heads=2, head_dim=128, d_ffn=1152, vocab_draft=3001,
                            vocab_target=4513, target_hidden=192, batch=1, K=5, ctx_lo=47,
                            ctx_hi=47, temps=(0.0,), sigma=0.05, vocab_map="inject",
                            shuffle_blocks=True),
    # One sequence over a 1100-position context: its draft steps merge 9 context splits
    # in the single-row O projection, its ingest passes through the split merge kernel.
    "p_single_splits": Workload(name="p_single_splits", cfg_id=20, dtype="bf16", n_layers=2,
                                d_model=256, n_q_heads=4, n_kv_heads=2, head_dim=128, d_ffn=512,
                                vocab_draft=3001, vocab_target=4513, target_hidden=192, batch=1,
                                K=5, ctx_lo=1100, ctx_hi=1100, temps=(1.0,), sigma=0.5,
                                vocab_map="inject"),
    # The same with 64-wide heads (8 of them in the merged row).
    "p_single_splits64": Workload(name="p_single_splits64", cfg_id=21, dtype="bf16", n_layers=2,
                                  d_model=256, n_q_heads=8, n_kv_heads=2, head_dim=64, d_ffn=512,
                                  vocab_draft=4001, vocab_target=4001, target_hidden=128, batch=1,
                                  K=6, ctx_lo=1100, ctx_hi=1100, temps=(0.7,), sigma=1.0,
                                  vocab_map="identity"),
    # Taps of 3 x 8192 columns: the pending ingest's tap projection (18 rows) has 24 K
    # splits, more than one round of the row kernel's split sum.
    "p_wide_taps": Workload(name="p_wide_taps", cfg_id=22, dtype="bf16", n_layers=2, d_model=256,
                            n_q_heads=4, n_kv_heads=2, head_dim=64, d_ffn=512, vocab_draft=3001,
                            vocab_target=3001, target_hidden=8192, batch=3, K=5, ctx_lo=20,
                            ctx_hi=44, temps=(1.0, 0.0, 0.7), sigma=0.5, shuffle_blocks=True),
    "p_inject": Workload(name="p_inject", cfg_id=14, dtype="bf16", n_layers=1, d_model=256,
                         n_q_heads=4, n_kv_heads=1, head_dim=128, d_ffn=512, vocab_draft=3001,
                         vocab_target=4513, target_hidden=192, batch=2, K=3, ctx_lo=1, ctx_hi=16,
                         temps=(0.7,), sigma=1.5, vocab_map="inject", shuffle_blocks=True),
    # block drafting: Llama-shaped body (no QK-norm), several sequences, mixed temperatures
    "p_block": Workload(name="p_block", cfg_id=18, dtype="bf16", n_layers=2, d_model=256,
                        n_q_heads=4, n_kv_heads=2, head_dim=64, d_ffn=640, qk_norm=0,
                        rope_theta=5.0e5, vocab_draft=4001, vocab_target=4001,
                        target_hidden=128, batch=3, K=7, ctx_lo=9, ctx_hi=40,
                        temps=(1.0, 0.0, 0.7), sigma=0.5, shuffle_blocks=True, drafting="block"),
    "p_block_single": Workload(name="p_block_single", cfg_id=19, dtype="bf16", n_layers=2,
                               d_model=384, n_q_heads=4, n_kv_heads=2, head_dim=128, d_ffn=1152,
                               vocab_draft=3001, vocab_target=4513, target_hidden=192, batch=1,
                               K=5, ctx_lo=47, ctx_hi=47, temps=(1.0,), sigma=0.3,
                               vocab_map="inject", shuffle_blocks=True, drafting="block"),
}


def get(name: str) -> Workload:
    if name in WORKLOADS:
        return WORKLOADS[name]
    if name in PARITY:
        return PARITY[name]
    raise KeyError(name)


def rng(w: Workload, stream: int, *sub: int) -> np.random.Generator:
    key = (int(w.cfg_id), int(w.variant), int(stream)) + tuple(int(s) for s in sub)
    return np.random.default_rng(np.random.SeedSequence(key))


def round_bf16(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bf16 value (ties to even); returns float32.

    Generated tensors declared bf16 are stored on this grid so that both the
    GPU (which holds them as bf16) and the oracle (which holds them as float
    values) see exactly the same numbers."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    bits = a.view(np.uint32)
    lsb = (bits >> np.uint32(16)) & np.uint32(1)
    rounded = (bits + np.uint32(0x7FFF) + lsb) & np.uint32(0xFFFF0000)
    return rounded.view(np.float32)


def _store(w: Workload, a: np.ndarray) -> np.ndarray:
    a = a.astype(np.float32, copy=False)
    return round_bf16(a) if w.dtype == "bf16" else a


# ---------------------------------------------------------------------------
# Weights
# ---------------------------------------------------------------------------
def weight_names(w: Workload) -> List[str]:
    names = ["embed", "w_c", "final_norm", "lm_head"]
    for l in range(w.n_layers):
        names += [f"layers.{l}.{n}" for n in ("in_norm", "w_qkv", "q_norm", "k_norm", "w_o",
                                              "post_norm", "w_gate", "w_up", "w_down")]
    return names


def weight_shapes(w: Workload) -> Dict[str, Tuple[int, ...]]:
    d, hd = w.d_model, w.head_dim
    s = {"embed": (w.vocab_target, d), "w_c": (d, w.tap_width), "final_norm": (d,),
         "lm_head": (w.vocab_draft, d)}
    for l in range(w.n_layers):
        p = f"layers.{l}."
        s[p + "in_norm"] = (d,)
        s[p + "w_qkv"] = (w.qkv_rows, 2 * d)      # columns [0, d): c-slot, [d, 2d): token
        s[p + "q_norm"] = (hd,)
        s[p + "k_norm"] = (hd,)
        s[p + "w_o"] = (d, w.n_q_heads * hd)
        s[p + "post_norm"] = (d,)
        s[p + "w_gate"] = (w.d_ffn, d)
        s[p + "w_up"] = (w.d_ffn, d)
        s[p + "w_down"] = (d, w.d_ffn)
    return s


def make_weights(w: Workload) -> Dict[str, np.ndarray]:
    """All drafter weights as float32 arrays (on the bf16 grid for bf16 workloads).

    Matrices and the embedding are N(0, 0.02); RMSNorm gains are 1, or
    1 + N(0, 0.1) when `gains == "normal"`.  With `expansion == "zero"` the
    c-slot columns of every W~_qkv are exactly zero (the adaptation-time
    initialisation of Section 3.3)."""
    shapes = weight_shapes(w)
    out = {}
    for i, name in enumerate(weight_names(w)):
        shp = shapes[name]
        g = rng(w, S_WEIGHTS, i)
        if len(shp) == 1:
            if w.gains == "normal":
                a = 1.0 + 0.1 * g.standard_normal(shp, dtype=np.float32)
            else:
                a = np.ones(shp, dtype=np.float32)
        else:
            a = g.standard_normal(shp, dtype=np.float32)
            a *= np.float32(0.02)
            if name.endswith("w_qkv") and w.expansion == "zero":
                a[:, : w.d_model] = 0.0
        out[name] = _store(w, a)
    return out


def make_d2t(w: Workload) -> np.ndarray:
    """Drafter-row -> target-id map (int32, -1 = unmapped).

    identity: V_d == V_T and d2t[i] = i.
    inject:   V_d <= V_T rows injected into a seeded subset of target ids.
    partial:  V_T of the V_d rows (a seeded choice) map onto a seeded
              permutation of all target ids; the rest are unmapped."""
    g = rng(w, S_VOCAB)
    vd, vt = w.vocab_draft, w.vocab_target
    if w.vocab_map == "identity":
        assert vd == vt
        return np.arange(vd, dtype=np.int32)
    if w.vocab_map == "inject":
        assert vd <= vt
        return g.choice(vt, size=vd, replace=False).astype(np.int32)
    if w.vocab_map == "partial":
        assert vd >= vt
        d2t = np.full(vd, -1, dtype=np.int32)
        rows = g.choice(vd, size=vt, replace=False)
        d2t[rows] = g.permutation(vt).astype(np.int32)
        return d2t
    raise ValueError(w.vocab_map)


# ---------------------------------------------------------------------------
# Sequences: contexts, prompts, synthetic context KV, paged block ids.
# ---------------------------------------------------------------------------
def context_lengths(w: Workload) -> np.ndarray:
    if w.ctx_lo == w.ctx_hi:
        return np.full(w.batch, w.ctx_lo, dtype=np.int64)
    return rng(w, S_CTX_LEN).integers(w.ctx_lo, w.ctx_hi + 1, size=w.batch)


def prompt_tokens(w: Workload, b: int, n: int) -> np.ndarray:
    return rng(w, S_PROMPT, b).integers(0, w.vocab_target, size=n).astype(np.int32)


def context_kv(w: Workload, b: int, n: int) -> Tuple[np.ndarray, np.ndarray]:
    """Synthetic post-RoPE keys and values for positions [0, n) of sequence b.

    Shapes [n_layers, n, n_kv_heads, head_dim]; N(0, 1) on the storage grid."""
    g = rng(w, S_CTX_KV, b)
    shp = (w.n_layers, n, w.n_kv_heads, w.head_dim)
    k = _store(w, g.standard_normal(shp, dtype=np.float32))
    v = _store(w, g.standard_normal(shp, dtype=np.float32))
    return k, v


def blocks_needed(w: Workload, capacity: int) -> int:
    return (capacity + w.kv_block - 1) // w.kv_block


def block_ids(w: Workload, n_blocks_per_seq: List[int]) -> List[np.ndarray]:
    """Physical KV-block ids per sequence: a partition of [0, sum) that is
    shuffled by seed when `shuffle_blocks`, else consecutive."""
    total = int(sum(n_blocks_per_seq))
    ids = np.arange(total, dtype=np.int32)
    if w.shuffle_blocks:
        ids = rng(w, S_BLOCKS).permutation(total).astype(np.int32)
    out, o = [], 0
    for n in n_blocks_per_seq:
        out.append(ids[o:o + n].copy())
        o += n
    return out


# ---------------------------------------------------------------------------
# Per-iteration inputs
# ---------------------------------------------------------------------------
def taps(w: Workload, it: int, b: int, rows: int) -> np.ndarray:
    """Target hidden-state taps for the new rows of sequence b at iteration `it`.

    Shape [rows, n_taps * H]; N(0, 1) on the storage grid.  Iteration -1 is
    the prefill (the prompt), whose first row is all-zero: position 0 has no
    predecessor, so its c-slot input is zero."""
    g = rng(w, S_TAPS, it + 1, b)
    t = _store(w, g.standard_normal((rows, w.tap_width), dtype=np.float32))
    return t


def uniforms(w: Workload, it: int, stream: int, shape) -> np.ndarray:
    """fp32 uniforms in [0, 1) on the 2^-24 grid (exact in fp32 and fp64)."""
    g = rng(w, stream, it + 1)
    return (g.integers(0, 1 << 24, size=shape).astype(np.float64) * 2.0 ** -24).astype(np.float32)


def u_draft(w: Workload, it: int) -> np.ndarray:
    return uniforms(w, it, S_U_DRAFT, (w.batch, max(w.K, 1)))


def u_accept(w: Workload, it: int) -> np.ndarray:
    return uniforms(w, it, S_U_ACC, (w.batch, max(w.K, 1)))


def u_bonus(w: Workload, it: int) -> np.ndarray:
    return uniforms(w, it, S_U_BONUS, (w.batch,))


def target_noise(w: Workload, it: int, b: int) -> np.ndarray:
    """N(0, 1) noise [K + 1, V_T] for the synthetic target logits of sequence b."""
    g = rng(w, S_NOISE, it + 1, b)
    return g.standard_normal((w.K + 1, w.vocab_target), dtype=np.float32)


def target_logits(w: Workload, draft_logits, d2t, noise):
    """Synthetic stand-in for the target's verify-pass logits of one sequence.

    draft_logits: [K, V_d] drafter logits (unmapped rows -inf); d2t: [V_d];
    noise: [K + 1, V_T].  Row k < K is the drafter row k carried to target ids
    plus sigma * noise; target ids no drafter row reaches take the mean of
    that row's mapped drafter logits as their base.  Row K (the bonus row)
    reuses drafter row K - 1 as its base with its own noise.  Works on numpy
    arrays or torch tensors (CPU or GPU) alike; returns float32."""
    try:
        import torch
        is_torch = isinstance(draft_logits, torch.Tensor)
    except ImportError:  # pragma: no cover
        is_torch = False
    K = w.K
    if is_torch:
        import torch
        dev = draft_logits.device
        dl = draft_logits.to(torch.float64)
        d2t_t = torch.as_tensor(d2t, device=dev, dtype=torch.int64)
        mapped = d2t_t >= 0
        base = torch.empty((K + 1, w.vocab_target), dtype=torch.float64, device=dev)
        rows = [dl[k] for k in range(K)] + [dl[K - 1]]
        for k, r in enumerate(rows):
            m = r[mapped]
            base[k].fill_(float(m.mean()))
            base[k, d2t_t[mapped]] = m
        nz = torch.as_tensor(noise, device=dev, dtype=torch.float64)
        return (base + w.sigma * nz).to(torch.float32)
    dl = np.asarray(draft_logits, dtype=np.float64)
    d2t = np.asarray(d2t)
    mapped = d2t >= 0
    base = np.empty((K + 1, w.vocab_target), dtype=np.float64)
    rows = [dl[k] for k in range(K)] + [dl[K - 1]]
    for k, r in enumerate(rows):
        m = r[mapped]
        base[k, :] = m.mean()
        base[k, d2t[mapped]] = m
    return (base + w.sigma * np.asarray(noise, dtype=np.float64)).astype(np.float32)


def tree_inputs(seed: int, V_T: int, n_nodes: int, topk: int, sigma: float):
    """A synthetic draft tree in the shape dynamic draft trees take, and target
    logits for it (inputs only; no verification arithmetic).

    Nodes are grown level by level: every frontier node gets up to `topk`
    children, and up to `topk` of the new nodes (chosen at random) form the next
    frontier, until there are n_nodes (parents before children).  Each row (root,
    then node i) has drafter-like logits N(0, 1.5); the children of a row carry
    its top-ranked tokens, best first, and the target row is those logits plus
    sigma * N(0, 1), so that the target often agrees with the first children.
    Returns parents [N] int32, tokens [N] int32, target logits [N + 1, V_T] fp32."""
    g = np.random.default_rng([0x7EE, seed])
    parents = []
    frontier = [-1]
    while len(parents) < n_nodes:
        new = []
        for f in frontier:
            for _ in range(topk):
                if len(parents) < n_nodes:
                    parents.append(f)
                    new.append(len(parents) - 1)
        if not new:
            break
        frontier = sorted(g.permutation(new)[:topk].tolist())
    parents = np.array(parents, dtype=np.int32)
    dl = g.standard_normal((n_nodes + 1, V_T)) * 1.5
    tokens = np.zeros(n_nodes, dtype=np.int32)
    rank, best = {}, {}
    for i, p in enumerate(parents):
        p = int(p)
        r = rank.get(p, 0)
        rank[p] = r + 1
        if p not in best:          # the row's topk best tokens, best first
            row = dl[p + 1]
            top = np.argpartition(-row, min(topk, V_T - 1))[:topk + 1]
            best[p] = top[np.argsort(-row[top], kind="stable")]
        tokens[i] = int(best[p][r])
    tl = dl + sigma * g.standard_normal((n_nodes + 1, V_T))
    return parents, tokens, tl.astype(np.float32)
