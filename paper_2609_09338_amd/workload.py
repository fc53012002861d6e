"""Drive libosprey on the seeded synthetic workloads (benchmark, smoke, tests).

Sequence b of a workload: positions [0, ctx_b - 1) are filled first (synthetic
post-RoPE keys/values through osprey_kv_append, or a K = 0 ingest of the
prompt); iteration 0 ingests prompt token ctx_b - 1 explicitly; iteration
i > 0 ingests the tokens the previous verification committed (pending mode,
no host synchronisation).  Taps, uniforms and temperatures come from `synth`.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Optional

import numpy as np

import synth

from . import _lib as L
from .binding import Drafter, make_config


def torch_dtype(w):
    import torch
    return torch.bfloat16 if w.dtype == "bf16" else torch.float32


def to_dev(a: np.ndarray, w, device):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).to(device=device, dtype=torch_dtype(w))


@dataclass
class Setup:
    w: "synth.Workload"
    drafter: Drafter
    ctx: np.ndarray
    blocks: List[np.ndarray]
    n_iters: int
    device: object
    temperature: object      # [B] float32 device tensor: the target's temperature
    draft_temperature: object  # [B] float32: the temperature drafts are drawn at


def capacity(w, ctx: int, n_iters: int) -> int:
    # pending ingests are bounded by K + 1 rows on the host: leave room for that bound
    return int(ctx) + (n_iters + 1) * (w.K + 1) + 2 * w.K + 1


def make_drafter(w, n_iters: int, device="cuda:0", weights=None) -> Setup:
    import torch
    weights = synth.make_weights(w) if weights is None else weights
    d2t = synth.make_d2t(w)
    ctx = synth.context_lengths(w)
    caps = [capacity(w, c, n_iters) for c in ctx]
    nblk = [synth.blocks_needed(w, c) for c in caps]
    blocks = synth.block_ids(w, nblk)
    prefill_rows = int(sum(c - 1 for c in ctx)) if w.prefill == "ingest" else 1
    cfg = make_config(n_layers=w.n_layers, d_model=w.d_model, n_q_heads=w.n_q_heads,
                      n_kv_heads=w.n_kv_heads, head_dim=w.head_dim, d_ffn=w.d_ffn,
                      vocab_draft=w.vocab_draft, vocab_target=w.vocab_target,
                      target_hidden=w.target_hidden, n_taps=w.n_taps,
                      dtype=L.OSPREY_BF16 if w.dtype == "bf16" else L.OSPREY_F32,
                      qk_norm=w.qk_norm, rms_eps=w.rms_eps, rope_theta=w.rope_theta,
                      max_batch=w.batch, max_k=w.K, max_seq_len=max(caps),
                      kv_block=w.kv_block, kv_num_blocks=int(sum(nblk)),
                      # (block drafting: new rows and the block's mask rows in one pass)
                      max_new_rows=max(prefill_rows, w.batch * (w.K + 1),
                                       w.batch * 2 * w.K if w.drafting == "block" else 0))
    tw = {k: to_dev(v, w, device) for k, v in weights.items()}
    dr = Drafter(cfg, tw, torch.from_numpy(d2t).to(device))
    temp = torch.tensor([w.temperature(b) for b in range(w.batch)], dtype=torch.float32,
                        device=device)
    temp_d = torch.tensor([w.draft_temperature(b) for b in range(w.batch)], dtype=torch.float32,
                          device=device)
    s = Setup(w, dr, ctx, blocks, n_iters, device, temp, temp_d)
    return s


def reset_sequences(s: Setup) -> None:
    """Empty every slot and fill positions [0, ctx_b - 1)."""
    import torch
    w, dr = s.w, s.drafter
    for b in range(w.batch):
        dr.seq_reset(b, s.blocks[b])
    if w.prefill == "kv":
        for b in range(w.batch):
            n = int(s.ctx[b]) - 1
            if n > 0:
                k, v = synth.context_kv(w, b, n)
                dr.kv_append(b, to_dev(k, w, s.device), to_dev(v, w, s.device))
    else:
        rows = [int(c) - 1 for c in s.ctx]
        sl = [b for b in range(w.batch) if rows[b] > 0]
        if sl:
            toks, taps = [], []
            for b in sl:
                toks.append(synth.prompt_tokens(w, b, int(s.ctx[b]))[: rows[b]])
                t = synth.taps(w, -1, b, rows[b])
                t[0] = 0.0
                taps.append(t)
            new_tokens = torch.from_numpy(np.concatenate(toks).astype(np.int32)).to(s.device)
            tp = to_dev(np.concatenate(taps), w, s.device)
            dr.draft_step(sl, 0, tp, s.draft_temperature[sl], n_new=[rows[b] for b in sl],
                          new_tokens=new_tokens, taps_stride=0)


@dataclass
class IterInputs:
    taps: object          # [B, K + 1, tap_w]
    u_draft: object       # [B, K]
    u_accept: object      # [B, K]
    u_bonus: object       # [B]
    new_tokens: Optional[object]  # iteration 0 only: [B]


def iter_inputs(s: Setup, it: int) -> IterInputs:
    import torch
    w = s.w
    taps = np.stack([synth.taps(w, it, b, w.K + 1) for b in range(w.batch)])
    f = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(s.device)
    nt = None
    if it == 0:
        nt = f(np.array([synth.prompt_tokens(w, b, int(s.ctx[b]))[-1] for b in range(w.batch)],
                        dtype=np.int32))
    return IterInputs(to_dev(taps, w, s.device), f(synth.u_draft(w, it)), f(synth.u_accept(w, it)),
                      f(synth.u_bonus(w, it)), nt)


@dataclass
class IterOutputs:
    drafts: object        # [B, K] int32
    logits: object        # [B, K, V_d] float32
    accept_len: object    # [B] int32
    mask: object          # [B, K] uint8
    tokens: object        # [B, K + 1] int32


def alloc_outputs(s: Setup) -> IterOutputs:
    import torch
    w, dev = s.w, s.device
    return IterOutputs(torch.empty((w.batch, w.K), dtype=torch.int32, device=dev),
                       torch.empty((w.batch, w.K, w.vocab_draft), dtype=torch.float32, device=dev),
                       torch.empty((w.batch,), dtype=torch.int32, device=dev),
                       torch.empty((w.batch, w.K), dtype=torch.uint8, device=dev),
                       torch.empty((w.batch, w.K + 1), dtype=torch.int32, device=dev))


def draft(s: Setup, it: int, inp: IterInputs, out: IterOutputs) -> None:
    w = s.w
    slots = list(range(w.batch))
    mask = synth.mask_token(w) if w.drafting == "block" else None
    if it == 0:
        s.drafter.draft_step(slots, w.K, inp.taps, s.draft_temperature, inp.u_draft,
                             n_new=[1] * w.batch, new_tokens=inp.new_tokens,
                             taps_stride=w.K + 1, draft_tokens=out.drafts,
                             draft_logits=out.logits, mask_token=mask)
    else:
        s.drafter.draft_step(slots, w.K, inp.taps, s.draft_temperature, inp.u_draft,
                             taps_stride=w.K + 1, draft_tokens=out.drafts,
                             draft_logits=out.logits, mask_token=mask)


def verify(s: Setup, inp: IterInputs, target_logits, out: IterOutputs) -> None:
    w = s.w
    s.drafter.verify(list(range(w.batch)), w.K, target_logits, s.temperature, inp.u_accept,
                     inp.u_bonus, out.accept_len, out.mask, out.tokens,
                     draft_temperature=s.draft_temperature)


def synthetic_target(s: Setup, it: int, draft_logits, d2t: Optional[np.ndarray] = None):
    """Target logits [B, K + 1, V_T] formed on the device from the drafter's
    logits of this iteration plus seeded noise (synth.target_logits)."""
    import torch
    w = s.w
    d2t = synth.make_d2t(w) if d2t is None else d2t
    rows = [synth.target_logits(w, draft_logits[b], d2t, synth.target_noise(w, it, b))
            for b in range(w.batch)]
    return torch.stack(rows).contiguous()
