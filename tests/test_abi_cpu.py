"""The C-ABI library without a GPU: it loads, exports every entry point the
header declares, and its host-only calls (configuration checks and sizing)
behave as documented.  No compute call runs here."""
import ctypes as C
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _ensure_built():
    from paper_2609_09338_amd import _lib
    if not os.path.exists(_lib.LIB_PATH):
        from paper_2609_09338_amd import build
        build.build(verbose=False)
    return _lib.load()


@pytest.fixture(scope="module")
def lib():
    return _ensure_built()


def _declared():
    src = open(os.path.join(ROOT, "include", "osprey.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(osprey_[a-z_]+)\s*\(", src)))


def test_every_declared_symbol_is_exported(lib):
    names = _declared()
    assert len(names) >= 17
    from paper_2609_09338_amd import _lib
    for n in names:
        assert hasattr(lib, n), n
        assert n in _lib.SIGNATURES, f"binding lacks {n}"


def _cfg(**kw):
    from paper_2609_09338_amd.binding import make_config
    base = dict(n_layers=2, d_model=1024, n_q_heads=16, n_kv_heads=8, head_dim=128, d_ffn=3072,
                vocab_draft=151936, vocab_target=151936, target_hidden=4096, dtype=1,
                max_batch=1, max_k=7, max_seq_len=4096, kv_num_blocks=256, max_new_rows=8)
    base.update(kw)
    return make_config(**base)


def test_config_validation_codes(lib):
    from paper_2609_09338_amd import binding as bd
    from paper_2609_09338_amd._lib import (OSPREY_E_INVALID, OSPREY_E_SHAPE, OSPREY_E_UNSUPPORTED,
                                           OSPREY_OK)
    assert bd.config_validate(_cfg()) == OSPREY_OK
    assert bd.config_validate(_cfg(d_model=1000)) == OSPREY_E_SHAPE
    assert bd.config_validate(_cfg(n_kv_heads=6)) == OSPREY_E_SHAPE
    assert bd.config_validate(_cfg(head_dim=96)) == OSPREY_E_UNSUPPORTED
    assert bd.config_validate(_cfg(kv_block=32)) == OSPREY_E_UNSUPPORTED
    assert bd.config_validate(_cfg(max_batch=0)) == OSPREY_E_INVALID
    assert bd.config_validate(_cfg(max_batch=257)) == OSPREY_E_INVALID
    assert bd.config_validate(_cfg(dtype=7)) == OSPREY_E_INVALID
    assert bd.config_validate(_cfg(target_hidden=4095)) == OSPREY_E_SHAPE
    assert "target_hidden" in bd.last_error()
    assert lib.osprey_config_validate(None) == OSPREY_E_INVALID


def test_pool_and_workspace_sizes(lib):
    from paper_2609_09338_amd import binding as bd
    c = _cfg()
    # [blocks][layers][k, v][kv heads][16 tokens x head_dim] bf16
    assert bd.kv_bytes(c) == 256 * 2 * 2 * 8 * 16 * 128 * 2
    assert bd.kv_bytes(_cfg(dtype=0)) == 2 * bd.kv_bytes(c)
    ws = bd.workspace_bytes(c)
    assert ws % 256 == 0
    # holds at least the stored drafter logits and the activations
    assert ws > 7 * 151936 * 4 + 8 * (2 * 1024 + 4096 + 3 * 2048 + 3072) * 4
    assert bd.workspace_bytes(_cfg(max_batch=8)) > ws
    assert bd.kv_bytes(_cfg(d_model=1000)) == 0 and bd.workspace_bytes(_cfg(d_model=1000)) == 0


@pytest.mark.skipif(__import__("torch").cuda.device_count() > 0,
                    reason="checks the no-device path; a GPU is present")
def test_init_without_a_device_reports_e_device(lib):
    from paper_2609_09338_amd import _lib as L
    c = _cfg()
    lw = (L.osprey_layer_weights * 2)()
    fake = 1 << 20
    for l in range(2):
        for f in ("in_norm", "w_qkv", "q_norm", "k_norm", "w_o", "post_norm", "w_gate", "w_up",
                  "w_down"):
            setattr(lw[l], f, fake)
    w = L.osprey_weights(fake, fake, fake, fake, fake, lw)
    h = C.c_void_p()
    kvb, wsb = lib.osprey_kv_bytes(C.byref(c)), lib.osprey_workspace_bytes(C.byref(c))
    rc = lib.osprey_draft_init(C.byref(c), C.byref(w), fake, kvb, fake, wsb, None, C.byref(h))
    assert rc == L.OSPREY_E_DEVICE
    assert "device" in lib.osprey_last_error().decode().lower()
    # argument errors are reported before the device is touched
    rc = lib.osprey_draft_init(C.byref(c), C.byref(w), fake + 8, kvb, fake, wsb, None, C.byref(h))
    assert rc == L.OSPREY_E_INVALID
    rc = lib.osprey_draft_init(C.byref(c), C.byref(w), fake, kvb - 1, fake, wsb, None, C.byref(h))
    assert rc == L.OSPREY_E_CAPACITY


def test_product_path_fails_loudly_without_the_library(tmp_path):
    from paper_2609_09338_amd import _lib as L
    saved = L._lib
    try:
        L._lib = None
        with pytest.raises(RuntimeError, match="not built"):
            L.load(str(tmp_path / "missing.so"))
    finally:
        L._lib = saved


def test_host_side_errors_of_the_newer_entry_points(lib):
    """The graph and no-allocation entry points refuse bad arguments before touching
    the device, with a message."""
    from paper_2609_09338_amd import _lib as L
    g = C.c_void_p()
    s, v = L.osprey_step_args(), L.osprey_verify_args()
    assert lib.osprey_graph_capture(None, C.byref(s), -1, C.byref(v), 64, C.byref(g)) == L.OSPREY_E_INVALID
    assert lib.osprey_graph_launch(None, None) == L.OSPREY_E_INVALID
    assert lib.osprey_graph_destroy(None) == L.OSPREY_OK
    a = L.osprey_verify_rows_args()
    a.batch, a.K = 65, 2
    assert lib.osprey_verify_rows_static(C.byref(a), C.c_void_p(16), 100, 100, None) == L.OSPREY_E_CAPACITY
    assert b"batch" in lib.osprey_last_error()
    a.batch, a.K = 4, 17
    assert lib.osprey_verify_rows_static(C.byref(a), C.c_void_p(16), 100, 100, None) == L.OSPREY_E_CAPACITY
    a.K = 2
    assert lib.osprey_verify_rows_static(C.byref(a), None, 100, 100, None) == L.OSPREY_E_INVALID
    assert lib.osprey_verify_rows_static(C.byref(a), C.c_void_p(16), 100, 262145, None) == L.OSPREY_E_CAPACITY
    # every pointer missing
    assert lib.osprey_verify_rows_static(C.byref(a), C.c_void_p(16), 100, 100, None) == L.OSPREY_E_INVALID
    assert lib.osprey_draft_destroy(None) == L.OSPREY_OK
