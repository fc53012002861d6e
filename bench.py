"""Benchmark of the Osprey draft-and-verify step on one MI355X.

    python bench.py [--gpus 1] [--steps 32] [--warmup 4] [--workload c2]
                    [--no-cpu-baseline] [--cpu-seconds 15]

A step is one iteration of the hot path for the whole batch: osprey_draft_step
(ingest of the tokens the previous verification committed + K autoregressive
draft steps) followed by osprey_verify.  The target model is not part of the
path: its logits for each iteration are synthetic (the drafter's logits plus
seeded noise) and, like every other input, are staged in HBM before the timed
region.  Because the whole path is deterministic, a first (untimed) pass
records the trajectory and its target logits; the timed pass replays it from
the same starting state.

The timed iterations run twice: as stream launches, and each iteration as one
HIP graph (osprey_graph_capture, captured before the timed region over that
iteration's staged inputs); the faster mode gives the headline and both are
reported.

Prints one JSON line: whole-job draft+verify tokens/s (sum over sequences of
accepted drafts + 1 per iteration, divided by the time of the draft_step and
verify calls), µs per draft step, the LM-head kernel and the attention against
the HBM roofline (timed with HIP events on the library's stream), and the CPU
oracle on a bounded sample (all cores and one thread).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=32)
    ap.add_argument("--warmup", type=int, default=4)
    ap.add_argument("--workload", default="c2")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-kernel-timing", action="store_true")
    ap.add_argument("--no-graph", action="store_true",
                    help="time stream launches only (no HIP-graph pass)")
    ap.add_argument("--long-contexts", default="16384,32768",
                    help="batch-1 attention is also timed at these contexts ('' = none)")
    ap.add_argument("--calibrate-copy-mib", type=int, default=0,
                    help="first copy a buffer of this many MiB device-to-device three times "
                         "(a reference for HBM traffic counters)")
    return ap.parse_args()


def copy_calibration(mib: int) -> None:
    """A plain device-to-device copy of known size: under rocprofv3 --pmc FETCH_SIZE /
    WRITE_SIZE its counters give the scale between counter units and bytes."""
    import torch
    n = mib * (1 << 20)
    src = torch.empty(n, dtype=torch.uint8, device="cuda:0").fill_(1)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst


def lm_head_bytes(w, rows: int) -> int:
    """Algorithmic HBM bytes of one LM-head launch: every weight byte once, the
    final-norm gain, the masked logits written and the vocabulary map read."""
    el = 2 if w.dtype == "bf16" else 4
    return w.vocab_draft * w.d_model * el + w.d_model * el + rows * w.vocab_draft * 4 \
        + w.vocab_draft * 4


def step_bytes(w, ctx_mean: float) -> dict:
    """Algorithmic bytes of one autoregressive draft step (all sequences)."""
    el = 2 if w.dtype == "bf16" else 4
    d, hd, L = w.d_model, w.head_dim, w.n_layers
    body = L * (w.qkv_rows * 2 * d + d * w.n_q_heads * hd + 3 * w.d_ffn * d + 2 * d + 2 * hd) * el
    lm = w.vocab_draft * d * el
    kv = w.batch * ctx_mean * L * 2 * w.n_kv_heads * hd * el
    return dict(body=body, lm=lm, kv=kv, total=body + lm + kv)


def iteration_bytes(w, sb: dict) -> int:
    """Algorithmic bytes of one iteration (all sequences): the ingest pass (W_c, the
    body, the LM head over each sequence's last row, the context), K - 1 autoregressive
    steps (the same without W_c), the K drafter logit rows written, and verification
    (the K + 1 target rows and one drafter row per sequence).  Block drafting: one pass
    (W_c, body, context, one LM head) and the same verification."""
    el = 2 if w.dtype == "bf16" else 4
    wc = w.tap_width * w.d_model * el
    verify = w.batch * ((w.K + 1) * w.vocab_target + w.vocab_draft) * 4
    logits = w.batch * w.K * w.vocab_draft * 4
    steps = 1 if w.drafting == "block" else w.K
    return int(wc + steps * sb["total"] + logits + verify)


def measured_traffic(workload: str, kernel: str = "lm_head"):
    """HBM bytes per launch of the LM head (or, kernel="attention", per attention pass)
    from the committed rocprofv3 --pmc summary, or None when there is none for this
    workload or the kernel's source changed since."""
    import hashlib
    try:
        t = json.load(open(os.path.join(ROOT, "profiles", "traffic.json")))[workload]
        if kernel != "lm_head":
            t = t[kernel]
        sha = hashlib.sha256(open(os.path.join(ROOT, t["source"]), "rb").read()).hexdigest()
    except (OSError, KeyError, ValueError):
        return None
    if not sha.startswith(t["sha256_prefix"]):
        return None
    return int(t["fetch_bytes"] + t["write_bytes"])


def run_gpu(args):
    import numpy as np
    import torch

    import synth
    from paper_2609_09338_amd import binding as BD
    from paper_2609_09338_amd import workload as WL

    w = synth.get(args.workload)
    n_it = args.warmup + args.steps
    dev = torch.device("cuda:0")
    s = WL.make_drafter(w, n_it, device=dev)
    WL.reset_sequences(s)
    d2t = synth.make_d2t(w)
    out = WL.alloc_outputs(s)

    # ---- record: inputs and synthetic target logits of every iteration ------------------
    gen = torch.Generator(device=dev)
    staged = []
    rec_accept = []
    for it in range(n_it):
        inp = WL.iter_inputs(s, it)
        WL.draft(s, it, inp, out)
        gen.manual_seed(1000003 * w.cfg_id + it)
        noise = torch.randn((w.batch, w.K + 1, w.vocab_target), generator=gen, device=dev)
        tl = torch.stack([synth.target_logits(w, out.logits[b], d2t, noise[b])
                          for b in range(w.batch)]).contiguous()
        del noise
        WL.verify(s, inp, tl, out)
        staged.append((inp, tl))
        rec_accept.append(out.accept_len.clone())
    torch.cuda.synchronize()
    rec_accept = torch.stack(rec_accept).cpu().numpy()

    def rewind():
        for b in range(w.batch):
            s.drafter.seq_truncate(b, int(s.ctx[b]) - 1)

    def replay(lo, hi, accept_out=None):
        for it in range(lo, hi):
            inp, tl = staged[it]
            WL.draft(s, it, inp, out)
            WL.verify(s, inp, tl, out)
            if accept_out is not None:
                accept_out.append(out.accept_len.clone())

    # ---- timed pass ---------------------------------------------------------------------
    rewind()
    replay(0, args.warmup)
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    acc = []
    t0 = time.perf_counter()
    ev0.record(s.drafter.stream)
    replay(args.warmup, n_it, acc)
    ev1.record(s.drafter.stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    gpu_ms = ev0.elapsed_time(ev1)
    got = torch.stack(acc).cpu().numpy()
    assert (got == rec_accept[args.warmup:]).all(), "replay diverged from the recorded trajectory"
    tokens = int((got + 1).sum())
    elapsed = max(gpu_ms / 1e3, 1e-9)
    res = dict(tokens=tokens, seconds=elapsed, wall=wall, mean_accept=float(got.mean()),
               modes={"stream": dict(seconds=elapsed, tokens=tokens)})
    if not args.no_graph and args.warmup >= 1:
        res["modes"]["graph"] = time_graph(s, w, staged, args.warmup, n_it, rec_accept, rewind,
                                           replay, out)
    res["trajectory"] = rec_accept
    # every attention pass of one pass over the iterations (the record pass, the timed
    # pass and the graph pass all run this same trajectory)
    passes = n_it * w.n_layers * (1 if w.drafting == "block" else w.K)
    res["attention_bytes_per_pass"] = attention_bytes(w, s.ctx, rec_accept, 0, n_it) / passes

    # ---- per-call and per-kernel timing: the same steps again, with HIP events on the
    #      library's stream; each event idles the stream for a few microseconds, so one
    #      replay brackets whole calls only and another the LM-head launches only -----------
    if not args.no_kernel_timing:
        kt = {}
        for fams in ((BD.KERNEL_DRAFT_STEP, BD.KERNEL_VERIFY), (BD.KERNEL_LM_HEAD,),
                     (BD.KERNEL_ATTENTION,)):
            rewind()
            replay(0, args.warmup)
            s.drafter.kernel_timing(fams)
            replay(args.warmup, n_it)
            torch.cuda.synchronize()
            for name, fam in (("lm_head", BD.KERNEL_LM_HEAD), ("verify", BD.KERNEL_VERIFY),
                              ("draft_step", BD.KERNEL_DRAFT_STEP),
                              ("attention", BD.KERNEL_ATTENTION)):
                if fam in fams:
                    kt[name] = s.drafter.kernel_time(fam)
            s.drafter.kernel_timing(())
        res["kernels"] = kt
        res["attention_bytes"] = attention_bytes(w, s.ctx, rec_accept, args.warmup, n_it)
        lens = [int(c) for c in args.long_contexts.split(",") if c.strip()]
        if lens and w.dtype == "bf16" and w.batch == 1 and w.drafting == "chain":
            res["attention_long"] = [time_attention_long(w, c) for c in lens]
        res["tree_verify"] = time_tree_verify(s, w)
        if w.dtype == "bf16" and w.K >= TREE_TOPK:
            rewind()
            res["tree_draft"] = time_tree_draft(s, w, float(np.mean(s.ctx)))
    assert s.drafter.device_errors() == 0
    res["ctx_mean"] = float(np.mean(s.ctx))
    return w, res


def time_graph(s, w, staged, warmup, n_it, rec_accept, rewind, replay, out):
    """The timed iterations again, each launched as one HIP graph (osprey_graph_capture
    of its pending draft call + verification over its staged inputs, captured before the
    timed region), on a stream of its own; the trajectory must be the recorded one."""
    import torch

    import synth
    dev, B = s.device, w.batch
    torch.cuda.synchronize()
    prev = s.drafter.stream
    st = torch.cuda.Stream(device=dev)
    s.drafter.set_stream(st)
    rewind()
    replay(0, warmup)
    accs = [torch.empty(B, dtype=torch.int32, device=dev) for _ in range(warmup, n_it)]
    mask = synth.mask_token(w) if w.drafting == "block" else None
    graphs = []
    for j, it in enumerate(range(warmup, n_it)):
        inp, tl = staged[it]
        graphs.append(s.drafter.capture_iteration(
            list(range(B)), w.K, inp.taps, s.draft_temperature, inp.u_draft, out.drafts,
            out.logits, tl, s.temperature, inp.u_accept, inp.u_bonus, accs[j], out.mask,
            out.tokens, max_context=int(s.drafter.cfg.max_seq_len), taps_stride=w.K + 1,
            mask_token=mask))
    st.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record(st)
    for g in graphs:
        g.launch()
    ev1.record(st)
    st.synchronize()
    ms = ev0.elapsed_time(ev1)
    got = torch.stack(accs).cpu().numpy()
    assert (got == rec_accept[warmup:]).all(), "graph replay diverged from the recorded trajectory"
    for g in graphs:
        g.close()
    s.drafter.set_stream(prev)
    return dict(seconds=max(ms / 1e3, 1e-9), tokens=int((got + 1).sum()))


def attention_bytes(w, ctx, traj, warmup: int, n_it: int) -> int:
    """Algorithmic bytes of every attention pass of the timed iterations: each sequence's
    context keys and values once per layer and pass.  Iteration `it` of sequence b
    commits L = ctx_b + sum_{j<it} (a_j + 1) positions; its ingest pass reads L of them,
    chain step k (1 <= k < K) reads L + k, a block pass L + K - 1."""
    import numpy as np
    el = 2 if w.dtype == "bf16" else 4
    tok = w.n_layers * 2 * w.n_kv_heads * w.head_dim * el
    total = 0
    for b in range(w.batch):
        L = int(ctx[b])
        for it in range(n_it):
            if it > 0:
                L += int(traj[it - 1][b]) + 1
            if it < warmup:
                continue
            if w.drafting == "block":
                total += (L + w.K - 1) * tok
            else:
                total += (L * w.K + w.K * (w.K - 1) // 2) * tok
    return int(total)


def time_attention_long(w, ctx_len: int, iters: int = 3):
    """Batch-1 attention (split pass + merge) of the drafter's AR steps at a long
    context: the same attention shape (heads, head dim, layers) with a small vocabulary
    (the attention does not depend on it), `iters` draft calls of K steps from the
    same committed prefix, HIP-event time per launch against each launch's context
    bytes."""
    import torch

    import synth
    from paper_2609_09338_amd import binding as BD
    from paper_2609_09338_amd import workload as WL
    wl = w.with_(name=f"{w.name}_ctx{ctx_len}", vocab_draft=4096, vocab_target=4096,
                 target_hidden=256, ctx_lo=ctx_len, ctx_hi=ctx_len)
    s = WL.make_drafter(wl, 1)
    WL.reset_sequences(s)
    out = WL.alloc_outputs(s)
    inp = WL.iter_inputs(s, 0)
    # (a drafted slot is verified before it is rewound; any target logits do)
    tl = torch.zeros((1, wl.K + 1, wl.vocab_target), dtype=torch.float32, device=s.device)
    WL.draft(s, 0, inp, out)
    WL.verify(s, inp, tl, out)
    torch.cuda.synchronize()
    el = 2 if wl.dtype == "bf16" else 4
    tok = 2 * wl.n_kv_heads * wl.head_dim * el
    s.drafter.kernel_timing((BD.KERNEL_ATTENTION,))
    nbytes = 0
    for _ in range(iters):
        s.drafter.seq_truncate(0, ctx_len - 1)
        WL.draft(s, 0, inp, out)
        WL.verify(s, inp, tl, out)
        # ingest pass: ctx positions; AR step k: ctx + k (per layer)
        nbytes += wl.n_layers * tok * (ctx_len * wl.K + wl.K * (wl.K - 1) // 2)
    torch.cuda.synchronize()
    ms, n = s.drafter.kernel_time(BD.KERNEL_ATTENTION)
    s.drafter.kernel_timing(())
    assert s.drafter.device_errors() == 0
    single_ms = ms / 8.0                # every timed pair ran 8 times between its events
    launches = n // 8
    gbs = nbytes / (single_ms * 1e-3) / 1e9
    s.drafter.close()
    del s
    torch.cuda.empty_cache()
    return dict(context=ctx_len, batch=1, us_per_launch=round(single_ms * 1e3 / max(launches, 1), 3),
                bytes_per_launch=int(nbytes / max(launches, 1)), achieved_gbs=round(gbs, 1),
                frac=round(gbs / HBM_PEAK_GBS, 4))


TREE_NODES, TREE_TOPK = 15, 4


def time_tree_verify(s, w, reps: int = 20):
    """Draft-tree verification (osprey_verify_tree) on synthetic 15-node, top-4 trees
    for every sequence of the batch at the workload's target vocabulary: per-call time
    from HIP events on the library's stream, against the bytes it must read (every
    target row once for its statistics, the last node's row again for the bonus)."""
    import numpy as np
    import torch

    import synth
    from paper_2609_09338_amd import binding as BD
    B, N, V = w.batch, TREE_NODES, w.vocab_target
    dev = s.device
    par, tok, tl = zip(*(synth.tree_inputs(b, V, N, TREE_TOPK, 0.3) for b in range(B)))
    T = lambda a: torch.from_numpy(np.ascontiguousarray(np.stack(a))).to(dev)
    g = np.random.default_rng(7)
    args = (T(tl), T(tok), T(par), torch.tensor([w.temperature(b) for b in range(B)], dtype=torch.float32, device=dev),
            torch.from_numpy((g.integers(0, 1 << 24, (B, N)) * 2.0 ** -24).astype(np.float32)).to(dev),
            torch.from_numpy((g.integers(0, 1 << 24, B) * 2.0 ** -24).astype(np.float32)).to(dev),
            torch.empty(B, dtype=torch.int32, device=dev), torch.empty((B, N), dtype=torch.int32, device=dev),
            torch.empty((B, N + 1), dtype=torch.int32, device=dev))
    s.drafter.verify_tree(*args)
    s.drafter.kernel_timing((BD.KERNEL_VERIFY,))
    for _ in range(reps):
        s.drafter.verify_tree(*args)
    torch.cuda.synchronize()
    ms, n = s.drafter.kernel_time(BD.KERNEL_VERIFY)
    s.drafter.kernel_timing(())
    us = ms * 1e3 / max(n, 1)
    nbytes = B * (N + 2) * V * 4
    return dict(nodes=N, topk=TREE_TOPK, batch=B, us_per_call=round(us, 2), bytes_per_call=nbytes,
                achieved_gbs=round(nbytes / (us * 1e-6) / 1e9, 1),
                frac=round(nbytes / (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4))


TREE_DEPTH = 4


def time_tree_draft(s, w, ctx_mean: float, reps: int = 10):
    """Draft-tree growth (osprey_draft_tree: ingest of one token per sequence, then a
    top-4, depth-4 tree of 15 nodes) for every sequence of the batch: per-call time
    from HIP events on the library's stream, against its algorithmic bytes (per depth
    every drafter weight and each sequence's context keys/values once, plus W_c for the
    ingest and the logits written).  Each call starts from the same committed prefix."""
    import numpy as np
    import torch

    import synth
    from paper_2609_09338_amd import binding as BD
    B, N, k, D = w.batch, TREE_NODES, TREE_TOPK, TREE_DEPTH
    dev = s.device
    taps = torch.zeros((B, w.tap_width), dtype=torch.bfloat16, device=dev)
    tok = torch.from_numpy(np.array([synth.prompt_tokens(w, b, int(s.ctx[b]))[-1]
                                     for b in range(B)], dtype=np.int32)).to(dev)
    tk = torch.empty((B, N), dtype=torch.int32, device=dev)
    pr = torch.empty((B, N), dtype=torch.int32, device=dev)

    def call():
        for b in range(B):
            s.drafter.seq_truncate(b, int(s.ctx[b]) - 1)
        s.drafter.draft_tree(list(range(B)), k, D, N, taps, s.temperature, tk, pr,
                             n_new=[1] * B, new_tokens=tok)

    call()
    s.drafter.kernel_timing((BD.KERNEL_DRAFT_STEP,))
    for _ in range(reps):
        call()
    torch.cuda.synchronize()
    ms, n = s.drafter.kernel_time(BD.KERNEL_DRAFT_STEP)
    s.drafter.kernel_timing(())
    for b in range(B):
        s.drafter.seq_truncate(b, int(s.ctx[b]) - 1)
    us = ms * 1e3 / max(n, 1)
    el = 2 if w.dtype == "bf16" else 4
    sb = step_bytes(w, ctx_mean)
    nbytes = int(D * sb["total"] + w.tap_width * w.d_model * el
                 + B * w.vocab_draft * 4 * (1 + (D - 1) * k))
    return dict(nodes=N, topk=k, depth=D, batch=B, us_per_call=round(us, 2),
                bytes_per_call=nbytes, achieved_gbs=round(nbytes / (us * 1e-6) / 1e9, 1),
                frac=round(nbytes / (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4))


def run_cpu_baseline(w, seconds: float):
    """The oracle, untuned, on one sequence of the same workload for ~`seconds`, twice:
    with every core of this process's affinity mask available to numpy's BLAS, and with
    one thread.  `cores` is the affinity mask's size; the all-core run is the headline
    figure and the one-thread run is reported next to it."""
    from threadpoolctl import threadpool_info, threadpool_limits

    from oracle import harness as OH
    cores = len(os.sched_getaffinity(0))
    dr = OH.build_drafter(w)

    def run(threads):
        with threadpool_limits(limits=threads):
            used = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
            t0 = time.perf_counter()
            tokens, iters = 0, 0
            for it in OH.run_sequence_timed(w, 0, 512, seconds, drafter=dr):
                tokens += it.result.accept_len + 1
                iters += 1
            dt = time.perf_counter() - t0
        return tokens / dt, iters, dt, used

    v_all, it_all, dt_all, used_all = run(cores)
    v_one, it_one, dt_one, _ = run(1)
    return dict(value=v_all, unit="tokens/s", cores=cores, kind="oracle",
                blas_threads=int(used_all),
                single_thread={"value": v_one, "unit": "tokens/s", "cores": 1,
                               "sample": f"{it_one} iteration(s), {dt_one:.1f} s"},
                sample=f"{it_all} iteration(s) of sequence 0 of workload {w.name} "
                       f"(K={w.K}, {w.K} drafter forward passes + verify each), "
                       f"{dt_all:.1f} s incl. setup, numpy float64")


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1",
                          "n_gpus": args.gpus}), flush=True)
        sys.exit(2)
    if args.calibrate_copy_mib > 0:
        copy_calibration(args.calibrate_copy_mib)
    w, r = run_gpu(args)
    K = args.steps
    # the faster launch mode is the headline; both are reported
    modes = r["modes"]
    mode = min(modes, key=lambda m: modes[m]["seconds"])
    seconds, tokens = modes[mode]["seconds"], modes[mode]["tokens"]
    ms_per_step = seconds * 1e3 / K
    value = tokens / seconds
    sb = step_bytes(w, r["ctx_mean"])
    it_bytes = iteration_bytes(w, sb)
    line = {
        "metric": "draft+verify tokens/s per GPU; µs per draft step at batch 1; % HBM peak",
        "value": round(value, 2), "unit": "tokens/s", "n_gpus": 1, "steps": K,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "storage_dtype": w.dtype,
        "data": "synthetic (seeded N(0,0.02) weights, N(0,1) taps and context KV, target "
                "logits = drafter logits + N(0, sigma))",
        "config": {"workload": f"{w.name}: {w.n_layers}-layer drafter d={w.d_model}, "
                               f"{w.n_q_heads}/{w.n_kv_heads} heads x {w.head_dim}, FFN {w.d_ffn}, "
                               f"V_d={w.vocab_draft}, V_T={w.vocab_target}, taps 3x{w.target_hidden}, "
                               f"batch {w.batch}, context {w.ctx_lo}"
                               + (f"-{w.ctx_hi}" if w.ctx_hi != w.ctx_lo else "")
                               + f", K={w.K}, T={list(w.temps)}"
                               + (", block drafting" if w.drafting == "block" else ""),
                   "batch": w.batch, "K": w.K},
        "mean_accepted_drafts": round(r["mean_accept"], 3),
        "tokens_timed": tokens,
        "launch_mode": mode,
        "launch_modes": {m: {"ms_per_step": round(v["seconds"] * 1e3 / K, 4),
                             "tokens_per_s": round(v["tokens"] / v["seconds"], 2)}
                         for m, v in modes.items()},
        "iteration_algorithmic_bytes": int(it_bytes),
        "attention_bytes_per_pass": int(r["attention_bytes_per_pass"]),
        "iteration_hbm_frac": round(it_bytes / (ms_per_step * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
    }
    kt = r.get("kernels")
    if kt:
        ds_ms, ds_n = kt["draft_step"]
        vf_ms, vf_n = kt["verify"]
        line["us_per_draft_step_call"] = round(ds_ms * 1e3 / max(ds_n, 1), 2)
        line["us_per_draft_token"] = round(ds_ms * 1e3 / max(ds_n, 1) / w.K, 2)
        line["us_per_verify"] = round(vf_ms * 1e3 / max(vf_n, 1), 2)
        lm_ms, lm_n = kt["lm_head"]
        lm_us = lm_ms * 1e3 / max(lm_n, 1)
        block = w.drafting == "block"
        # (block drafting: one head launch over every sequence's K block rows)
        bytes_launch = lm_head_bytes(w, w.batch * (w.K if block else 1))
        ach = bytes_launch / (lm_us * 1e-6) / 1e9
        line["roofline"] = {"bound": "hbm", "kernel": "LM head (final RMSNorm + vocabulary GEMV "
                            "+ masked logits + softmax block statistics)",
                            "achieved": round(ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                            "frac": round(ach / HBM_PEAK_GBS, 4),
                            "traffic": measured_traffic(args.workload),
                            "bytes_per_launch": bytes_launch, "us_per_launch": round(lm_us, 3),
                            "launches": lm_n, "timing": "HIP events on the library stream, "
                            "8 back-to-back launches per event pair"}
        if block:
            # a block call: one pass over the new and the block rows (tap projection, the
            # body's weights and each sequence's context once), one LM head over the
            # block rows, the logits written
            el = 2 if w.dtype == "bf16" else 4
            call = (w.tap_width * w.d_model * el + sb["body"] + sb["kv"] + sb["lm"]
                    + w.batch * w.K * w.vocab_draft * 4)
            call_us = ds_ms * 1e3 / max(ds_n, 1)
            line["draft_call_algorithmic_bytes"] = int(call)
            line["draft_call_hbm_frac"] = round(call / (call_us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)
        else:
            line["ar_step_algorithmic_bytes"] = int(sb["total"])
            ar_us = ds_ms * 1e3 / max(ds_n, 1) / w.K
            line["draft_token_hbm_frac"] = round(sb["total"] / (ar_us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)
        at_ms, at_n = kt["attention"]
        if at_n:
            # every timed attention pass ran 8 times between its events
            at_s = at_ms / 8.0 * 1e-3
            at_gbs = r["attention_bytes"] / at_s / 1e9
            line["attention_roofline"] = {
                "bound": "hbm", "kernel": "attention (paged split pass, and the split merge kernel "
                "where one runs: passes whose O projection merges the splits launch none), every "
                "pass of the timed iterations", "achieved": round(at_gbs, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(at_gbs / HBM_PEAK_GBS, 4),
                "traffic": measured_traffic(args.workload, "attention"),
                "us_per_launch": round(at_s * 1e6 / max(at_n // 8, 1), 3),
                "bytes_per_launch": int(r["attention_bytes"] / max(at_n // 8, 1)),
                "launches": at_n // 8}
        if "attention_long" in r:
            line["attention_long_context"] = r["attention_long"]
        line["tree_verify"] = r["tree_verify"]
        if "tree_draft" in r:
            line["tree_draft"] = r["tree_draft"]
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = run_cpu_baseline(w, args.cpu_seconds)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
