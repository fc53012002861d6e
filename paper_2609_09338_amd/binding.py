"""Python binding of libosprey: the C-ABI calls under the same names, taking
torch tensors for device buffers.  Argument marshalling only -- every step of
the draft-and-verify path runs in the HIP kernels of the library.  PyTorch
provides device memory and the stream."""
from __future__ import annotations

import ctypes as C
from typing import Dict, Optional, Sequence

from . import _lib as L
from ._lib import osprey_config, osprey_layer_weights, osprey_weights  # noqa: F401

LAYER_FIELDS = ("in_norm", "w_qkv", "q_norm", "k_norm", "w_o", "post_norm", "w_gate", "w_up",
                "w_down")


class OspreyError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{L.STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


def _lib():
    return L.load()


def _check(rc: int) -> None:
    if rc != 0:
        raise OspreyError(rc, _lib().osprey_last_error().decode())


def _ptr(t) -> Optional[int]:
    return None if t is None else int(t.data_ptr())


def _need(t, numel: int, dtype, name: str) -> None:
    """Refuse a device buffer that is smaller than the call will touch."""
    if t is None:
        return
    if not t.is_cuda or not t.is_contiguous():
        raise ValueError(f"{name}: need a contiguous device tensor")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name}: dtype {t.dtype}, expected {dtype}")
    if t.numel() < numel:
        raise ValueError(f"{name}: {t.numel()} elements, the call needs {numel}")


def _i32_array(xs: Sequence[int]):
    arr = (C.c_int32 * len(xs))(*[int(x) for x in xs])
    return arr


def make_config(**kw) -> osprey_config:
    c = osprey_config()
    defaults = dict(n_taps=3, qk_norm=1, rms_eps=1e-6, rope_theta=1e6, kv_block=16, max_new_rows=1)
    for k, v in {**defaults, **kw}.items():
        setattr(c, k, v)
    return c


def config_validate(cfg: osprey_config) -> int:
    return int(_lib().osprey_config_validate(C.byref(cfg)))


def kv_bytes(cfg: osprey_config) -> int:
    return int(_lib().osprey_kv_bytes(C.byref(cfg)))


def workspace_bytes(cfg: osprey_config) -> int:
    return int(_lib().osprey_workspace_bytes(C.byref(cfg)))


def last_error() -> str:
    return _lib().osprey_last_error().decode()


def expected_weight_shapes(cfg) -> Dict[str, tuple]:
    """Shapes of the tensors include/osprey.h describes (osprey_weights)."""
    d, hd = cfg.d_model, cfg.head_dim
    s = {"embed": (cfg.vocab_target, d), "w_c": (d, cfg.n_taps * cfg.target_hidden),
         "final_norm": (d,), "lm_head": (cfg.vocab_draft, d)}
    for l in range(cfg.n_layers):
        p = f"layers.{l}."
        s.update({p + "in_norm": (d,), p + "w_qkv": ((cfg.n_q_heads + 2 * cfg.n_kv_heads) * hd, 2 * d),
                  p + "w_o": (d, cfg.n_q_heads * hd), p + "post_norm": (d,),
                  p + "w_gate": (cfg.d_ffn, d), p + "w_up": (cfg.d_ffn, d),
                  p + "w_down": (d, cfg.d_ffn)})
        if cfg.qk_norm:
            s.update({p + "q_norm": (hd,), p + "k_norm": (hd,)})
    return s


class Drafter:
    """A drafter handle plus the device buffers it was given.

    weights: name -> device tensor (dtype of the config), names as
    "embed", "w_c", "final_norm", "lm_head", "layers.{l}.{field}".
    d2t: int32 device tensor [V_d]."""

    def __init__(self, cfg: osprey_config, weights: Dict[str, "object"], d2t, stream=None):
        import torch
        self.cfg = cfg
        self.torch = torch
        _check(_lib().osprey_config_validate(C.byref(cfg)))
        dev = d2t.device
        want = torch.bfloat16 if cfg.dtype == L.OSPREY_BF16 else torch.float32
        self._wdtype = want
        self.weights = {}
        for k, t in weights.items():
            if t.dtype != want or not t.is_contiguous() or t.device != dev:
                raise ValueError(f"weight {k}: need a contiguous {want} tensor on {dev}")
            self.weights[k] = t
        if d2t.dtype != torch.int32 or not d2t.is_contiguous() or d2t.numel() != cfg.vocab_draft:
            raise ValueError("d2t must be a contiguous int32 tensor of vocab_draft entries")
        shapes = expected_weight_shapes(cfg)
        for k, shp in shapes.items():
            if k not in self.weights:
                raise ValueError(f"missing weight {k}")
            if tuple(self.weights[k].shape) != shp:
                raise ValueError(f"weight {k}: shape {tuple(self.weights[k].shape)}, expected {shp}")
        self.d2t = d2t
        self.kv = torch.empty(kv_bytes(cfg), dtype=torch.uint8, device=dev)
        self.ws = torch.empty(workspace_bytes(cfg), dtype=torch.uint8, device=dev)
        self._layers = (osprey_layer_weights * cfg.n_layers)()
        for l in range(cfg.n_layers):
            for f in LAYER_FIELDS:
                t = self.weights.get(f"layers.{l}.{f}")
                setattr(self._layers[l], f, _ptr(t))
        self._w = osprey_weights(_ptr(self.weights["embed"]), _ptr(self.weights["w_c"]),
                                 _ptr(self.weights["final_norm"]), _ptr(self.weights["lm_head"]),
                                 _ptr(d2t), self._layers)
        self.stream = stream if stream is not None else torch.cuda.current_stream(dev)
        h = C.c_void_p()
        _check(_lib().osprey_draft_init(C.byref(cfg), C.byref(self._w), _ptr(self.kv),
                                        self.kv.numel(), _ptr(self.ws), self.ws.numel(),
                                        C.c_void_p(self.stream.cuda_stream), C.byref(h)))
        self.h = h
        self._keep = []

    # -- sequences --------------------------------------------------------------------
    def seq_reset(self, slot: int, block_ids: Sequence[int]) -> None:
        arr = _i32_array(block_ids)
        _check(_lib().osprey_seq_reset(self.h, slot, arr, len(block_ids)))

    def kv_append(self, slot: int, k, v) -> None:
        n = int(k.shape[1])
        c = self.cfg
        need = c.n_layers * n * c.n_kv_heads * c.head_dim
        _need(k, need, self._wdtype, "k")
        _need(v, need, self._wdtype, "v")
        _check(_lib().osprey_kv_append(self.h, slot, n, _ptr(k), _ptr(v)))

    def seq_truncate(self, slot: int, length: int) -> None:
        _check(_lib().osprey_seq_truncate(self.h, slot, length))

    def seq_length(self, slot: int) -> int:
        out = C.c_int32()
        _check(_lib().osprey_seq_length(self.h, slot, C.byref(out)))
        return int(out.value)

    # -- the step ---------------------------------------------------------------------
    def draft_step(self, slots, K: int, taps, temperature, u_draft=None, n_new=None,
                   new_tokens=None, taps_stride: int = 0, draft_tokens=None,
                   draft_logits=None, mask_token=None) -> None:
        """Ingest the new rows and propose K drafts: a chain of K steps
        (osprey_draft_step), or one block (osprey_draft_block) when mask_token is given."""
        torch, c = self.torch, self.cfg
        B = len(slots)
        tap_w = c.n_taps * c.target_hidden
        rows = B * taps_stride if taps_stride > 0 else int(sum(n_new or []))
        _need(taps, rows * tap_w, self._wdtype, "taps")
        _need(temperature, B, torch.float32, "temperature")
        _need(u_draft, B * K, torch.float32, "u_draft")
        _need(draft_tokens, B * K, torch.int32, "draft_tokens")
        _need(draft_logits, B * K * c.vocab_draft, torch.float32, "draft_logits")
        if n_new is not None:
            _need(new_tokens, int(sum(n_new)), torch.int32, "new_tokens")
        a, keep = _step_args(slots, K, taps, temperature, u_draft, n_new, new_tokens,
                             taps_stride, draft_tokens, draft_logits)
        if mask_token is None:
            _check(_lib().osprey_draft_step(self.h, C.byref(a)))
        else:
            _check(_lib().osprey_draft_block(self.h, C.byref(a), int(mask_token)))

    def draft_tree(self, slots, topk: int, depth: int, n_nodes: int, taps, temperature,
                   tokens, parents, n_new, new_tokens, taps_stride: int = 0,
                   scores=None) -> None:
        """Ingest the new rows and grow a draft tree (osprey_draft_tree); tokens and
        parents [B, n_nodes] int32 outputs, scores [B, n_nodes] float64 (optional)."""
        torch, c = self.torch, self.cfg
        B = len(slots)
        tap_w = c.n_taps * c.target_hidden
        rows = B * taps_stride if taps_stride > 0 else int(sum(n_new))
        _need(taps, rows * tap_w, self._wdtype, "taps")
        _need(temperature, B, torch.float32, "temperature")
        _need(new_tokens, int(sum(n_new)), torch.int32, "new_tokens")
        _need(tokens, B * n_nodes, torch.int32, "tokens")
        _need(parents, B * n_nodes, torch.int32, "parents")
        if scores is not None:
            _need(scores, B * n_nodes, torch.float64, "scores")
        a = L.osprey_step_args()
        a.batch = B
        a.K = 0
        sl = _i32_array(slots)
        a.slots = C.cast(sl, C.POINTER(C.c_int32))
        nn = _i32_array(n_new)
        a.n_new = C.cast(nn, C.POINTER(C.c_int32))
        a.new_tokens = _ptr(new_tokens)
        a.taps = _ptr(taps)
        a.taps_stride = taps_stride
        a.temperature = _ptr(temperature)
        t = L.osprey_tree_args()
        t.topk = topk
        t.depth = depth
        t.n_nodes = n_nodes
        t.tokens = _ptr(tokens)
        t.parents = _ptr(parents)
        t.scores = _ptr(scores) if scores is not None else None
        _check(_lib().osprey_draft_tree(self.h, C.byref(a), C.byref(t)))

    def verify(self, slots, K: int, target_logits, temperature, u_accept, u_bonus,
               accept_len, accept_mask, out_tokens, draft_temperature=None) -> None:
        torch, c = self.torch, self.cfg
        B = len(slots)
        _need(target_logits, B * (K + 1) * c.vocab_target, torch.float32, "target_logits")
        _need(temperature, B, torch.float32, "temperature")
        _need(u_accept, B * K, torch.float32, "u_accept")
        _need(u_bonus, B, torch.float32, "u_bonus")
        _need(accept_len, B, torch.int32, "accept_len")
        _need(accept_mask, B * K, torch.uint8, "accept_mask")
        _need(out_tokens, B * (K + 1), torch.int32, "out_tokens")
        _need(draft_temperature, B, torch.float32, "draft_temperature")
        a, keep = _verify_args(slots, K, target_logits, temperature, u_accept, u_bonus,
                               accept_len, accept_mask, out_tokens, draft_temperature)
        _check(_lib().osprey_verify(self.h, C.byref(a)))

    # -- one iteration as a HIP graph ---------------------------------------------------
    def set_stream(self, stream) -> None:
        """Enqueue subsequent calls on `stream` (a torch.cuda.Stream)."""
        _check(_lib().osprey_set_stream(self.h, C.c_void_p(stream.cuda_stream)))
        self.stream = stream

    def capture_iteration(self, slots, K: int, taps, draft_temperature, u_draft, draft_tokens,
                          draft_logits, target_logits, temperature, u_accept, u_bonus,
                          accept_len, accept_mask, out_tokens, max_context: int,
                          taps_stride: int, mask_token=None) -> "IterationGraph":
        """osprey_graph_capture: a pending-mode draft call and its verification recorded
        as one HIP graph over exactly these buffers (see IterationGraph)."""
        torch, c = self.torch, self.cfg
        B = len(slots)
        _need(taps, B * taps_stride * c.n_taps * c.target_hidden, self._wdtype, "taps")
        _need(draft_temperature, B, torch.float32, "draft_temperature")
        _need(u_draft, B * K, torch.float32, "u_draft")
        _need(draft_tokens, B * K, torch.int32, "draft_tokens")
        _need(draft_logits, B * K * c.vocab_draft, torch.float32, "draft_logits")
        _need(target_logits, B * (K + 1) * c.vocab_target, torch.float32, "target_logits")
        _need(temperature, B, torch.float32, "temperature")
        _need(u_accept, B * K, torch.float32, "u_accept")
        _need(u_bonus, B, torch.float32, "u_bonus")
        _need(accept_len, B, torch.int32, "accept_len")
        _need(accept_mask, B * K, torch.uint8, "accept_mask")
        _need(out_tokens, B * (K + 1), torch.int32, "out_tokens")
        sa, k1 = _step_args(slots, K, taps, draft_temperature, u_draft, None, None, taps_stride,
                            draft_tokens, draft_logits)
        va, k2 = _verify_args(slots, K, target_logits, temperature, u_accept, u_bonus,
                              accept_len, accept_mask, out_tokens, draft_temperature)
        g = C.c_void_p()
        _check(_lib().osprey_graph_capture(self.h, C.byref(sa),
                                           -1 if mask_token is None else int(mask_token),
                                           C.byref(va), int(max_context), C.byref(g)))
        # the graph holds raw pointers: keep the tensors alive with it
        return IterationGraph(self, g, (taps, draft_temperature, u_draft, draft_tokens,
                                        draft_logits, target_logits, temperature, u_accept,
                                        u_bonus, accept_len, accept_mask, out_tokens))

    def verify_rows(self, K: int, target_logits, draft_logits, draft_tokens, temperature,
                    u_accept, u_bonus, accept_len, accept_mask, out_tokens,
                    draft_temperature=None) -> None:
        torch, c = self.torch, self.cfg
        B = int(target_logits.shape[0])
        _need(target_logits, B * (K + 1) * c.vocab_target, torch.float32, "target_logits")
        _need(draft_logits, B * K * c.vocab_draft, torch.float32, "draft_logits")
        _need(draft_tokens, B * K, torch.int32, "draft_tokens")
        _need(temperature, B, torch.float32, "temperature")
        _need(u_accept, B * K, torch.float32, "u_accept")
        _need(u_bonus, B, torch.float32, "u_bonus")
        _need(accept_len, B, torch.int32, "accept_len")
        _need(accept_mask, B * K, torch.uint8, "accept_mask")
        _need(out_tokens, B * (K + 1), torch.int32, "out_tokens")
        _need(draft_temperature, B, torch.float32, "draft_temperature")
        a = L.osprey_verify_rows_args()
        a.batch = B
        a.K = K
        a.target_logits = _ptr(target_logits)
        a.draft_logits = _ptr(draft_logits)
        a.draft_tokens = _ptr(draft_tokens)
        a.temperature = _ptr(temperature)
        a.u_accept = _ptr(u_accept)
        a.u_bonus = _ptr(u_bonus)
        a.accept_len = _ptr(accept_len)
        a.accept_mask = _ptr(accept_mask)
        a.out_tokens = _ptr(out_tokens)
        a.draft_temperature = _ptr(draft_temperature)
        _check(_lib().osprey_verify_rows(self.h, C.byref(a)))

    def verify_tree(self, target_logits, tokens, parents, temperature, u_accept, u_bonus,
                    accept_len, accept_path, out_tokens) -> None:
        """Lossless verification of a draft tree (osprey_verify_tree): target_logits
        [B, N + 1, V_T], tokens / parents / u_accept [B, N], outputs accept_len [B],
        accept_path [B, N], out_tokens [B, N + 1]."""
        torch, c = self.torch, self.cfg
        B = int(target_logits.shape[0])
        N = int(target_logits.shape[1]) - 1
        _need(target_logits, B * (N + 1) * c.vocab_target, torch.float32, "target_logits")
        _need(tokens, B * N, torch.int32, "tokens")
        _need(parents, B * N, torch.int32, "parents")
        _need(temperature, B, torch.float32, "temperature")
        _need(u_accept, B * N, torch.float32, "u_accept")
        _need(u_bonus, B, torch.float32, "u_bonus")
        _need(accept_len, B, torch.int32, "accept_len")
        _need(accept_path, B * N, torch.int32, "accept_path")
        _need(out_tokens, B * (N + 1), torch.int32, "out_tokens")
        a = L.osprey_verify_tree_args()
        a.batch = B
        a.n_nodes = N
        a.target_logits = _ptr(target_logits)
        a.tokens = _ptr(tokens)
        a.parents = _ptr(parents)
        a.temperature = _ptr(temperature)
        a.u_accept = _ptr(u_accept)
        a.u_bonus = _ptr(u_bonus)
        a.accept_len = _ptr(accept_len)
        a.accept_path = _ptr(accept_path)
        a.out_tokens = _ptr(out_tokens)
        _check(_lib().osprey_verify_tree(self.h, C.byref(a)))

    # -- diagnostics ------------------------------------------------------------------
    def device_errors(self) -> int:
        f = C.c_uint32()
        _check(_lib().osprey_device_errors(self.h, C.byref(f)))
        return int(f.value)

    def kernel_timing(self, families=()) -> None:
        """Event timing of the given kernel families (KERNEL_*); () disables it."""
        mask = 0
        for f in families:
            mask |= 1 << int(f)
        _check(_lib().osprey_kernel_timing(self.h, mask))

    def kernel_time(self, family: int):
        ms, n = C.c_double(), C.c_int64()
        _check(_lib().osprey_kernel_time(self.h, family, C.byref(ms), C.byref(n)))
        return float(ms.value), int(n.value)

    def close(self) -> None:
        if getattr(self, "h", None):
            _lib().osprey_draft_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def verify_rows_static(K: int, target_logits, draft_logits, draft_tokens, temperature, u_accept,
                       u_bonus, accept_len, accept_mask, out_tokens, d2t, vocab_target: int,
                       stream=None, draft_temperature=None) -> None:
    """osprey_verify_rows_static: osprey_verify_rows with no handle; its scratch is the
    library's fixed device array (limits: batch 64, K 16, vocabularies 262144)."""
    import torch
    B = int(target_logits.shape[0])
    V_d = int(d2t.numel())
    _need(target_logits, B * (K + 1) * vocab_target, torch.float32, "target_logits")
    _need(draft_logits, B * K * V_d, torch.float32, "draft_logits")
    _need(draft_tokens, B * K, torch.int32, "draft_tokens")
    _need(temperature, B, torch.float32, "temperature")
    _need(u_accept, B * K, torch.float32, "u_accept")
    _need(u_bonus, B, torch.float32, "u_bonus")
    _need(accept_len, B, torch.int32, "accept_len")
    _need(accept_mask, B * K, torch.uint8, "accept_mask")
    _need(out_tokens, B * (K + 1), torch.int32, "out_tokens")
    _need(draft_temperature, B, torch.float32, "draft_temperature")
    _need(d2t, V_d, torch.int32, "d2t")
    a = L.osprey_verify_rows_args()
    a.batch = B
    a.K = K
    a.target_logits = _ptr(target_logits)
    a.draft_logits = _ptr(draft_logits)
    a.draft_tokens = _ptr(draft_tokens)
    a.temperature = _ptr(temperature)
    a.u_accept = _ptr(u_accept)
    a.u_bonus = _ptr(u_bonus)
    a.accept_len = _ptr(accept_len)
    a.accept_mask = _ptr(accept_mask)
    a.out_tokens = _ptr(out_tokens)
    a.draft_temperature = _ptr(draft_temperature)
    st = stream if stream is not None else torch.cuda.current_stream()
    _check(_lib().osprey_verify_rows_static(C.byref(a), _ptr(d2t), V_d, int(vocab_target),
                                            C.c_void_p(st.cuda_stream)))


class IterationGraph:
    """A captured iteration (osprey_graph_*): launch() enqueues it on the drafter's
    stream; close() releases it (after the stream has finished with it)."""

    def __init__(self, drafter: Drafter, g, tensors):
        self.drafter, self.g, self._tensors = drafter, g, tensors

    def launch(self) -> None:
        _check(_lib().osprey_graph_launch(self.drafter.h, self.g))

    def close(self) -> None:
        if getattr(self, "g", None):
            _lib().osprey_graph_destroy(self.g)
            self.g = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def _step_args(slots, K, taps, temperature, u_draft, n_new, new_tokens, taps_stride,
               draft_tokens, draft_logits):
    a = L.osprey_step_args()
    a.batch = len(slots)
    a.K = K
    sl = _i32_array(slots)
    a.slots = C.cast(sl, C.POINTER(C.c_int32))
    nn = None
    if n_new is not None:
        nn = _i32_array(n_new)
        a.n_new = C.cast(nn, C.POINTER(C.c_int32))
    a.new_tokens = _ptr(new_tokens)
    a.taps = _ptr(taps)
    a.taps_stride = taps_stride
    a.temperature = _ptr(temperature)
    a.u_draft = _ptr(u_draft)
    a.draft_tokens = _ptr(draft_tokens)
    a.draft_logits = _ptr(draft_logits)
    return a, (sl, nn)


def _verify_args(slots, K, target_logits, temperature, u_accept, u_bonus, accept_len,
                 accept_mask, out_tokens, draft_temperature):
    a = L.osprey_verify_args()
    a.batch = len(slots)
    a.K = K
    sl = _i32_array(slots)
    a.slots = C.cast(sl, C.POINTER(C.c_int32))
    a.target_logits = _ptr(target_logits)
    a.temperature = _ptr(temperature)
    a.u_accept = _ptr(u_accept)
    a.u_bonus = _ptr(u_bonus)
    a.accept_len = _ptr(accept_len)
    a.accept_mask = _ptr(accept_mask)
    a.out_tokens = _ptr(out_tokens)
    a.draft_temperature = _ptr(draft_temperature)
    return a, (sl,)


KERNEL_LM_HEAD, KERNEL_ATTENTION, KERNEL_VERIFY, KERNEL_DRAFT_STEP, KERNEL_QKV = range(5)
