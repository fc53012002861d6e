"""osprey_verify_rows_static (no handle, no caller workspace: its scratch is the
library's fixed device array) against osprey_verify_rows on the same inputs, through
the C ABI: accepted lengths, masks and tokens bit for bit, on two calls in a row (the
second smaller, so the array holds the first call's contents when it starts), and its
size limits refused before anything is enqueued."""
import numpy as np
import pytest
import torch

import synth
from oracle import sampling as OS

pytestmark = pytest.mark.gpu


def _require_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_09338_amd import _lib
    _lib.load()


def _case(V_d, V_T, vmap, B, K, seed):
    from paper_2609_09338_amd import workload as WL
    w = synth.Workload(name=f"na_{V_d}", cfg_id=360 + V_d % 89, dtype="bf16", n_layers=1, d_model=64,
                       n_q_heads=1, n_kv_heads=1, head_dim=64, d_ffn=64, vocab_draft=V_d,
                       vocab_target=V_T, target_hidden=8, batch=B, K=K, ctx_lo=1, ctx_hi=1,
                       vocab_map=vmap)
    s = WL.make_drafter(w, 1)
    d2t = synth.make_d2t(w)
    rng = np.random.default_rng(seed)
    temps = np.array([[0.0, 0.7, 1.0, 1.3][b % 4] for b in range(B)], dtype=np.float32)
    temps_d = np.array([[0.0, 0.7, 1.0, 0.5][(b // 2) % 4] for b in range(B)], dtype=np.float32)
    dl = (rng.standard_normal((B, K, V_d)) * 1.5).astype(np.float32)
    dl[:, :, d2t < 0] = -np.inf
    u_d = rng.integers(0, 1 << 24, (B, K)) * 2.0 ** -24
    drafts = np.array([[d2t[OS.pick(dl[b, k], float(temps_d[b]), float(u_d[b, k]))]
                        for k in range(K)] for b in range(B)], dtype=np.int32).reshape(B, K)
    tl = np.zeros((B, K + 1, V_T), dtype=np.float32)
    for b in range(B):
        tl[b] = synth.target_logits(w.with_(sigma=0.5), dl[b], d2t,
                                    rng.standard_normal((K + 1, V_T)).astype(np.float32))
    u_a = (rng.integers(0, 1 << 24, (B, K)) * 2.0 ** -24).astype(np.float32)
    u_b = (rng.integers(0, 1 << 24, B) * 2.0 ** -24).astype(np.float32)
    dev = s.device
    T = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    ins = (T(tl), T(dl), T(drafts), T(temps), T(u_a), T(u_b))
    return s, ins, T(temps_d), T(d2t.astype(np.int32)), V_T


def test_static_verify_equals_verify_rows_on_two_calls():
    _require_gpu()
    from paper_2609_09338_amd import binding as BD
    accepted = 0
    for V_d, V_T, vmap, B, K, seed in ((151936, 151936, "identity", 48, 6, 1),
                                       (3001, 4513, "inject", 5, 3, 2)):
        print(f"[no_alloc] V_d {V_d} V_T {V_T} batch {B} K {K}", flush=True)
        s, ins, temps_d, d2t, V_T = _case(V_d, V_T, vmap, B, K, seed)
        dev = s.device
        outs = []
        for fn in ("rows", "static"):
            al = torch.full((B,), -7, dtype=torch.int32, device=dev)
            mk = torch.full((B, K), 7, dtype=torch.uint8, device=dev)
            ot = torch.full((B, K + 1), -7, dtype=torch.int32, device=dev)
            if fn == "rows":
                s.drafter.verify_rows(K, *ins, al, mk, ot, draft_temperature=temps_d)
            else:
                BD.verify_rows_static(K, *ins, al, mk, ot, d2t, V_T,
                                      stream=torch.cuda.current_stream(), draft_temperature=temps_d)
            torch.cuda.synchronize()
            outs.append((al.cpu(), mk.cpu(), ot.cpu()))
        for x, y in zip(*outs):
            assert torch.equal(x, y), (V_d, x, y)
        accepted += int(outs[0][0].sum())
        assert s.drafter.device_errors() == 0
    assert accepted > 0


def test_static_verify_refuses_sizes_beyond_its_array():
    _require_gpu()
    import ctypes as C
    from paper_2609_09338_amd import _lib as L
    lib = L.load()
    a = L.osprey_verify_rows_args()
    a.batch, a.K = 65, 2
    assert lib.osprey_verify_rows_static(C.byref(a), C.c_void_p(16), 100, 100, None) == L.OSPREY_E_CAPACITY
    a.batch, a.K = 4, 17
    assert lib.osprey_verify_rows_static(C.byref(a), C.c_void_p(16), 100, 100, None) == L.OSPREY_E_CAPACITY
    a.K = 2
    assert lib.osprey_verify_rows_static(C.byref(a), C.c_void_p(16), 262145, 100, None) == L.OSPREY_E_CAPACITY
    assert b"262144" in lib.osprey_last_error()
