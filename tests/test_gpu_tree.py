"""GPU parity of draft-tree verification (osprey_verify_tree) against the oracle.

Synthetic trees grown level by level with the drafter-like rows' top tokens as
children (synth.tree_inputs), target rows close to those rows, a mix of
temperatures per sequence (0, 0.7, 1.0, 1.3), and edge cases: an empty tree,
chains, the 64-node maximum, a duplicate sibling token and a node whose parent
is not an earlier node (device error bit 5; the node is unreachable on both
sides).  Accepted lengths, paths and tokens must be bit-exact except where a
decision is flagged as a near tie (tests/parity.py, tree_flags).
"""
import numpy as np
import pytest
import torch

import synth
from oracle.tree import verify_tree as o_verify_tree

from . import parity

pytestmark = pytest.mark.gpu


def _require_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_09338_amd import _lib
    _lib.load()


def _say(*a):
    print(*a, flush=True)


def _run(s, tl, tokens, parents, temps, u_a, u_b):
    dev = s.device
    T = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    B, N1 = tl.shape[0], tl.shape[1]
    N = N1 - 1
    al = torch.full((B,), -7, dtype=torch.int32, device=dev)
    ap = torch.full((B, max(N, 1)), -7, dtype=torch.int32, device=dev)
    ot = torch.full((B, N + 1), -7, dtype=torch.int32, device=dev)
    s.drafter.verify_tree(T(tl), T(tokens) if N else None, T(parents) if N else None, T(temps),
                          T(u_a) if N else None, T(u_b), al, ap if N else None, ot)
    torch.cuda.synchronize()
    return al.cpu().numpy(), ap.cpu().numpy()[:, :N], ot.cpu().numpy(), s.drafter.device_errors()


@pytest.mark.parametrize("V_T,N,topk,sigma", [(997, 15, 4, 0.3), (151936, 15, 4, 0.3),
                                               (4513, 64, 3, 0.1), (151936, 5, 1, 0.3),
                                               (997, 0, 4, 0.3), (4513, 24, 8, 1.0)])
def test_verify_tree_matches_oracle(V_T, N, topk, sigma):
    _require_gpu()
    from paper_2609_09338_amd import workload as WL
    _say(f"[verify_tree] V_T {V_T} N {N} topk {topk}")
    w = synth.Workload(name=f"vt_{V_T}_{N}", cfg_id=400 + N, dtype="bf16", n_layers=1,
                       d_model=64, n_q_heads=1, n_kv_heads=1, head_dim=64, d_ffn=64,
                       vocab_draft=V_T, vocab_target=V_T, target_hidden=8, batch=16, K=5,
                       ctx_lo=1, ctx_hi=1, vocab_map="identity")
    s = WL.make_drafter(w, 1)
    B = w.batch
    rng = np.random.default_rng(N * 131 + V_T)
    tl = np.zeros((B, N + 1, V_T), dtype=np.float32)
    tokens = np.zeros((B, N), dtype=np.int32)
    parents = np.zeros((B, N), dtype=np.int32)
    for b in range(B):
        parents[b], tokens[b], tl[b] = synth.tree_inputs(1000 * N + b, V_T, N, topk, sigma)
    temps = np.array([[0.0, 0.7, 1.0, 1.3][b % 4] for b in range(B)], dtype=np.float32)
    u_a = (rng.integers(0, 1 << 24, (B, N)) * 2.0 ** -24).astype(np.float32)
    u_b = (rng.integers(0, 1 << 24, B) * 2.0 ** -24).astype(np.float32)
    al, ap, ot, err = _run(s, tl, tokens, parents, temps, u_a, u_b)
    assert err == 0
    flagged = accepted = 0
    for b in range(B):
        r = o_verify_tree(tl[b], tokens[b], parents[b], float(temps[b]), u_a[b], float(u_b[b]))
        A = r.accept_len
        exp_path = np.full(N, -1)
        exp_path[:A] = r.path
        exp_tok = np.full(N + 1, -1)
        exp_tok[:A + 1] = r.tokens
        same = al[b] == A and np.array_equal(ap[b], exp_path) and np.array_equal(ot[b], exp_tok)
        if not same:
            assert parity.tree_flags(r, tl[b], tokens[b], parents[b], float(temps[b]), u_a[b],
                                     float(u_b[b])), (b, al[b], A, ap[b], exp_path, ot[b], exp_tok)
            flagged += 1
        accepted += A
    assert flagged <= 2
    if N > 0 and sigma <= 0.3:
        assert accepted > 0


def test_verify_tree_duplicate_and_invalid_parent():
    _require_gpu()
    from paper_2609_09338_amd import workload as WL
    _say("[verify_tree] duplicate token, invalid parent")
    V_T, N = 997, 6
    w = synth.Workload(name="vt_edge", cfg_id=499, dtype="bf16", n_layers=1, d_model=64,
                       n_q_heads=1, n_kv_heads=1, head_dim=64, d_ffn=64, vocab_draft=V_T,
                       vocab_target=V_T, target_hidden=8, batch=4, K=5, ctx_lo=1, ctx_hi=1,
                       vocab_map="identity")
    s = WL.make_drafter(w, 1)
    B = w.batch
    rng = np.random.default_rng(3)
    tl = (rng.standard_normal((B, N + 1, V_T)) * 0.5).astype(np.float32)
    tl[:, :, 5] += 6.0          # the target strongly prefers token 5 at every node
    tokens = np.array([[7, 5, 5, 9, 5, 5]] * B, dtype=np.int32)   # duplicate 5 among the root's
    parents = np.array([[-1, -1, -1, 1, 1, 3]] * B, dtype=np.int32)
    parents[1, 4] = 4           # not an earlier node: unreachable, error bit 5
    temps = np.array([0.0, 1.0, 1.0, 0.7], dtype=np.float32)
    u_a = (rng.integers(0, 1 << 24, (B, N)) * 2.0 ** -24).astype(np.float32)
    u_b = (rng.integers(0, 1 << 24, B) * 2.0 ** -24).astype(np.float32)
    al, ap, ot, err = _run(s, tl, tokens, parents, temps, u_a, u_b)
    assert err == (1 << 5)
    for b in range(B):
        par = parents[b].copy()
        par[(par < -1) | (par >= np.arange(N))] = -2
        r = o_verify_tree(tl[b], tokens[b], par, float(temps[b]), u_a[b], float(u_b[b]))
        assert al[b] == r.accept_len and list(ap[b][:r.accept_len]) == list(r.path), b
        assert list(ot[b][:r.accept_len + 1]) == list(r.tokens), b
        assert 2 not in list(ap[b])          # the duplicate sibling is never accepted


# ----------------------------------------------------------------------------------------
# growing trees (osprey_draft_tree) against the oracle's tree growth
# ----------------------------------------------------------------------------------------
def _path_keys(tokens, parents):
    """Each node's path from the root as a tuple of tokens (identifies a node across
    two trees whose generation orders differ)."""
    keys = []
    for i in range(len(tokens)):
        k, j = [], i
        while j >= 0:
            k.append(int(tokens[j]))
            j = int(parents[j])
        keys.append(tuple(k[::-1]))
    return keys


@pytest.mark.parametrize("wl,topk,depth,n_nodes,seqs", [("p_qwen_small", 3, 4, 12, None),
                                                        ("p_single128", 4, 3, 15, None),
                                                        ("p_partial", 2, 5, 9, None),
                                                        ("p_greedy_draft", 5, 2, 30, None),
                                                        # the benchmark's trees at full size
                                                        ("c2", 4, 4, 15, None),
                                                        ("c5", 4, 4, 15, [5, 63])])
def test_draft_tree_matches_oracle(wl, topk, depth, n_nodes, seqs):
    """Two tree steps per sequence: the first ingests the last prompt token, the
    second the tokens that following each tree's first children for two levels
    commits, plus one more (the same on both sides).  The GPU tree must be valid
    (parents earlier, the root's children first at depth 1), its scores within 2e-2
    of the oracle's on every node both trees hold, and the trees (tokens, parents)
    identical unless one of the oracle's selections had a margin below four times
    that measured score error (a near tie that another rounding may break).  Full-size
    workloads run the whole batch on the GPU; the oracle follows the sampled sequences
    (sequences of a batch are independent)."""
    _require_gpu()
    from oracle import harness as OH
    from oracle.tree import draft_tree as o_draft_tree
    from paper_2609_09338_amd import workload as WL
    _say(f"[draft_tree] {wl} topk {topk} depth {depth} nodes {n_nodes}")
    w = synth.get(wl)
    s = WL.make_drafter(w, 3)
    WL.reset_sequences(s)
    dr = OH.build_drafter(w)
    B, dev = w.batch, s.device
    picked = list(range(B)) if seqs is None else seqs
    oseq = {b: OH.start_sequence(w, dr, b, 3) for b in picked}
    new_tok = [np.array([synth.prompt_tokens(w, b, int(s.ctx[b]))[-1]], dtype=np.int64)
               for b in range(B)]
    flagged = compared = 0
    max_err = 0.0
    for step in range(2):
        taps = np.stack([synth.taps(w, step, b, w.K + 1) for b in range(B)])
        n_new = [len(t) for t in new_tok]
        tok_d = torch.from_numpy(np.concatenate(new_tok).astype(np.int32)).to(dev)
        tk = torch.full((B, n_nodes), -7, dtype=torch.int32, device=dev)
        pr = torch.full((B, n_nodes), -7, dtype=torch.int32, device=dev)
        sc = torch.full((B, n_nodes), 7.0, dtype=torch.float64, device=dev)
        s.drafter.draft_tree(list(range(B)), topk, depth, n_nodes, WL.to_dev(taps, w, dev),
                             s.temperature, tk, pr, n_new=n_new, new_tokens=tok_d,
                             taps_stride=w.K + 1, scores=sc)
        torch.cuda.synchronize()
        assert s.drafter.device_errors() == 0
        tk, pr, sc = tk.cpu().numpy(), pr.cpu().numpy(), sc.cpu().numpy()
        nxt = [np.array([int(tk[b, 0])], dtype=np.int64) for b in range(B)]
        for b in picked:
            t = o_draft_tree(dr, oseq[b], new_tok[b], taps[b][: n_new[b]].astype(np.float64),
                             topk, depth, n_nodes)
            compared += 1
            # a valid tree: parents earlier, scores non-increasing along every path
            assert all(-1 <= pr[b, i] < i for i in range(n_nodes)), pr[b]
            assert all(pr[b, i] < 0 or sc[b, i] <= sc[b, pr[b, i]] for i in range(n_nodes))
            assert np.all(tk[b] >= 0) and np.all(tk[b] < w.vocab_target)
            gk = dict(zip(_path_keys(tk[b], pr[b]), sc[b]))
            ok = dict(zip(_path_keys(t.tokens, t.parents), t.scores))
            common = set(gk) & set(ok)
            assert common, (wl, step, b)
            err = max(abs(gk[k] - ok[k]) for k in common)
            assert err <= 2e-2, (wl, step, b, err)
            max_err = max(max_err, err)
            if not (np.array_equal(tk[b], t.tokens) and np.array_equal(pr[b], t.parents)):
                near = parity.tree_near_tie_keys(t, 4.0 * err + 1e-9)
                assert parity.tree_mismatch_excused(_path_keys(tk[b], pr[b]),
                                                    _path_keys(t.tokens, t.parents), near), \
                    (wl, step, b, tk[b], t.tokens, pr[b], t.parents, t.min_gap, err)
                flagged += 1
            # commit: the first child of each node for two levels, then the root's first child
            path, cur = [], -1
            while len(path) < 2:
                kids = np.flatnonzero(t.parents == cur)
                if len(kids) == 0:
                    break
                cur = int(kids[0])
                path.append(int(t.tokens[cur]))
            nxt[b] = np.array(path + [int(t.tokens[0])], dtype=np.int64)
        new_tok = nxt
    _say(f"[draft_tree] {wl}: compared {compared} flagged {flagged} max score error {max_err:.3g}")
    assert flagged <= max(1, compared // 5)
