"""ctypes declarations of the C ABI in include/osprey.h (argument marshalling only)."""
from __future__ import annotations

import ctypes as C
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
# OSPREY_LIB names another build of the same library (the host-sanitized one of the CPU
# tests); there is no fallback either way
LIB_PATH = os.environ.get("OSPREY_LIB") or os.path.join(_HERE, "libosprey.so")

OSPREY_OK, OSPREY_E_INVALID, OSPREY_E_SHAPE, OSPREY_E_CAPACITY, OSPREY_E_STATE, \
    OSPREY_E_DEVICE, OSPREY_E_UNSUPPORTED = 0, -1, -2, -3, -4, -5, -6
OSPREY_F32, OSPREY_BF16 = 0, 1

STATUS_NAMES = {0: "OK", -1: "E_INVALID", -2: "E_SHAPE", -3: "E_CAPACITY", -4: "E_STATE",
                -5: "E_DEVICE", -6: "E_UNSUPPORTED"}


class osprey_config(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("d_model", C.c_int32), ("n_q_heads", C.c_int32),
                ("n_kv_heads", C.c_int32), ("head_dim", C.c_int32), ("d_ffn", C.c_int32),
                ("vocab_draft", C.c_int32), ("vocab_target", C.c_int32),
                ("target_hidden", C.c_int32), ("n_taps", C.c_int32), ("dtype", C.c_int32),
                ("qk_norm", C.c_int32), ("rms_eps", C.c_float), ("rope_theta", C.c_float),
                ("max_batch", C.c_int32), ("max_k", C.c_int32), ("max_seq_len", C.c_int32),
                ("kv_block", C.c_int32), ("kv_num_blocks", C.c_int32),
                ("max_new_rows", C.c_int32)]


class osprey_layer_weights(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in ("in_norm", "w_qkv", "q_norm", "k_norm", "w_o",
                                          "post_norm", "w_gate", "w_up", "w_down")]


class osprey_weights(C.Structure):
    _fields_ = [("embed", C.c_void_p), ("w_c", C.c_void_p), ("final_norm", C.c_void_p),
                ("lm_head", C.c_void_p), ("d2t", C.c_void_p),
                ("layers", C.POINTER(osprey_layer_weights))]


class osprey_step_args(C.Structure):
    _fields_ = [("batch", C.c_int32), ("K", C.c_int32), ("slots", C.POINTER(C.c_int32)),
                ("n_new", C.POINTER(C.c_int32)), ("new_tokens", C.c_void_p), ("taps", C.c_void_p),
                ("taps_stride", C.c_int32), ("temperature", C.c_void_p), ("u_draft", C.c_void_p),
                ("draft_tokens", C.c_void_p), ("draft_logits", C.c_void_p)]


class osprey_verify_args(C.Structure):
    _fields_ = [("batch", C.c_int32), ("K", C.c_int32), ("slots", C.POINTER(C.c_int32)),
                ("target_logits", C.c_void_p), ("temperature", C.c_void_p),
                ("u_accept", C.c_void_p), ("u_bonus", C.c_void_p), ("accept_len", C.c_void_p),
                ("accept_mask", C.c_void_p), ("out_tokens", C.c_void_p),
                ("draft_temperature", C.c_void_p)]


class osprey_verify_rows_args(C.Structure):
    _fields_ = [("batch", C.c_int32), ("K", C.c_int32), ("target_logits", C.c_void_p),
                ("draft_logits", C.c_void_p), ("draft_tokens", C.c_void_p),
                ("temperature", C.c_void_p), ("u_accept", C.c_void_p), ("u_bonus", C.c_void_p),
                ("accept_len", C.c_void_p), ("accept_mask", C.c_void_p),
                ("out_tokens", C.c_void_p), ("draft_temperature", C.c_void_p)]


class osprey_verify_tree_args(C.Structure):
    _fields_ = [("batch", C.c_int32), ("n_nodes", C.c_int32), ("target_logits", C.c_void_p),
                ("tokens", C.c_void_p), ("parents", C.c_void_p), ("temperature", C.c_void_p),
                ("u_accept", C.c_void_p), ("u_bonus", C.c_void_p), ("accept_len", C.c_void_p),
                ("accept_path", C.c_void_p), ("out_tokens", C.c_void_p)]


class osprey_tree_args(C.Structure):
    _fields_ = [("topk", C.c_int32), ("depth", C.c_int32), ("n_nodes", C.c_int32),
                ("tokens", C.c_void_p), ("parents", C.c_void_p), ("scores", C.c_void_p)]


_P = C.c_void_p
_H = C.c_void_p
SIGNATURES = {
    "osprey_config_validate": (C.c_int, [C.POINTER(osprey_config)]),
    "osprey_kv_bytes": (C.c_size_t, [C.POINTER(osprey_config)]),
    "osprey_workspace_bytes": (C.c_size_t, [C.POINTER(osprey_config)]),
    "osprey_draft_init": (C.c_int, [C.POINTER(osprey_config), C.POINTER(osprey_weights), _P,
                                    C.c_size_t, _P, C.c_size_t, _P, C.POINTER(_H)]),
    "osprey_seq_reset": (C.c_int, [_H, C.c_int32, C.POINTER(C.c_int32), C.c_int32]),
    "osprey_kv_append": (C.c_int, [_H, C.c_int32, C.c_int32, _P, _P]),
    "osprey_seq_truncate": (C.c_int, [_H, C.c_int32, C.c_int32]),
    "osprey_seq_length": (C.c_int, [_H, C.c_int32, C.POINTER(C.c_int32)]),
    "osprey_draft_step": (C.c_int, [_H, C.POINTER(osprey_step_args)]),
    "osprey_verify": (C.c_int, [_H, C.POINTER(osprey_verify_args)]),
    "osprey_verify_rows": (C.c_int, [_H, C.POINTER(osprey_verify_rows_args)]),
    "osprey_verify_tree": (C.c_int, [_H, C.POINTER(osprey_verify_tree_args)]),
    "osprey_verify_rows_static": (C.c_int, [C.POINTER(osprey_verify_rows_args), _P, C.c_int32,
                                            C.c_int32, _P]),
    "osprey_draft_tree": (C.c_int, [_H, C.POINTER(osprey_step_args), C.POINTER(osprey_tree_args)]),
    "osprey_draft_block": (C.c_int, [_H, C.POINTER(osprey_step_args), C.c_int32]),
    "osprey_device_errors": (C.c_int, [_H, C.POINTER(C.c_uint32)]),
    "osprey_kernel_timing": (C.c_int, [_H, C.c_int32]),
    "osprey_kernel_time": (C.c_int, [_H, C.c_int32, C.POINTER(C.c_double),
                                     C.POINTER(C.c_int64)]),
    "osprey_set_stream": (C.c_int, [_H, _P]),
    "osprey_graph_capture": (C.c_int, [_H, C.POINTER(osprey_step_args), C.c_int32,
                                       C.POINTER(osprey_verify_args), C.c_int32, C.POINTER(_P)]),
    "osprey_graph_launch": (C.c_int, [_H, _P]),
    "osprey_graph_destroy": (C.c_int, [_P]),
    "osprey_draft_destroy": (C.c_int, [_H]),
    "osprey_last_error": (C.c_char_p, []),
}

_lib = None


def load(path: str = LIB_PATH) -> C.CDLL:
    """Load libosprey.so and declare its signatures.  Raises if it is not built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built: run `python -m paper_2609_09338_amd.build` "
                           "(the HIP library is required; there is no fallback)")
    lib = C.CDLL(path)
    for name, (res, args) in SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib
