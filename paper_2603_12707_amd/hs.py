"""Thin ctypes binding of libhs (include/hs.h).

Argument marshalling only: every step of prefill and decode runs in the HIP
kernels of libhs.so.  torch tensors supply device memory and the current HIP
stream.  The library is loaded from this package directory; if it is missing
the import fails loudly (there is no fallback path).
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
# HS_LIBRARY names another build of the same library (the host-sanitizer
# build of the tests); by default the in-tree libhs.so
LIB_PATH = os.environ.get("HS_LIBRARY") or os.path.join(HERE, "libhs.so")

HS_OK, HS_E_INVALID, HS_E_CAPACITY, HS_E_BUFFER, HS_E_STATE, HS_E_DEVICE = 0, -1, -2, -3, -4, -5
HS_F32, HS_F16, HS_BF16 = 0, 1, 2
HS_ROPE_1D, HS_ROPE_M3 = 0, 1

# every symbol include/hs.h declares
EXPORTS = ("hs_last_error", "hs_kv_bytes", "hs_model_create", "hs_model_free", "hs_kv_alloc", "hs_kv_free",
           "hs_prefill_embeddings", "hs_decode_step", "hs_model_status", "hs_kv_lengths", "hs_kv_write",
           "hs_kv_read", "hs_kv_set_length", "hs_replay_kernels", "hs_packed_bytes", "hs_pack_matrix", "hs_pack_matrix_heads", "hs_kv_sync",
           "hs_prefill_batch", "hs_model_reserve_rows", "hs_kv_pool_create", "hs_kv_admit", "hs_kv_release",
           "hs_kv_pool_blocks", "hs_handoff_create", "hs_handoff_free", "hs_handoff_push", "hs_handoff_pop",
           "hs_handoff_pending", "hs_stream_read", "hs_decode_step_static")

# projection matrices the library reads in its packed layout
PACKED = ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down", "lm_head")

HS_K_NAMES = ("embed", "qkv", "attn", "combine", "oproj", "gateup", "down", "head", "argmax")


class HsError(RuntimeError):
    def __init__(self, func: str, code: int, msg: str):
        super().__init__(f"{func} failed with status {code}: {msg}")
        self.code = code


class hs_config(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32), ("n_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("ffn_dim", ctypes.c_int32),
                ("vocab", ctypes.c_int32), ("rope_theta", ctypes.c_float), ("rms_eps", ctypes.c_float),
                ("rope_kind", ctypes.c_int32), ("mrope_section", ctypes.c_int32 * 3),
                ("qkv_bias", ctypes.c_int32), ("dtype", ctypes.c_int32)]


class hs_layer_weights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("attn_norm", "wq", "wk", "wv", "bq", "bk", "bv", "wo", "mlp_norm",
                                                 "w_gate", "w_up", "w_down")]


class hs_weights(ctypes.Structure):
    _fields_ = [("embed", ctypes.c_void_p), ("final_norm", ctypes.c_void_p), ("lm_head", ctypes.c_void_p),
                ("layers", ctypes.POINTER(hs_layer_weights))]


_lib = None


def lib() -> ctypes.CDLL:
    """Loads libhs.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    # torch ships its own HIP runtime under the same soname as the system one;
    # importing it first makes libhs.so bind to that runtime instead of
    # loading a second copy into the process
    import torch  # noqa: F401
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with paper_2603_12707_amd/build.py "
                          "(or __graft_entry__.build()); there is no fallback implementation")
    L = ctypes.CDLL(LIB_PATH)
    P, I32, I64, U64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64
    L.hs_last_error.restype = ctypes.c_char_p
    L.hs_last_error.argtypes = []
    sig = {
        "hs_kv_bytes": [ctypes.POINTER(hs_config), I64, I64, ctypes.POINTER(U64), ctypes.POINTER(U64)],
        "hs_model_create": [ctypes.POINTER(hs_config), ctypes.POINTER(hs_weights), I32, I32, ctypes.POINTER(P)],
        "hs_model_free": [P],
        "hs_kv_alloc": [P, I32, P, P, P, U64, ctypes.POINTER(P)],
        "hs_kv_free": [P],
        "hs_prefill_embeddings": [P, P, I32, P, P, I32, P, P, P, P],
        "hs_prefill_batch": [P, P, I32, P, P, P, P, P, P, P, P],
        "hs_model_reserve_rows": [P, I64],
        "hs_kv_pool_create": [P, I32, I32, P, U64, ctypes.POINTER(P)],
        "hs_kv_admit": [P, I32, I32, I32, P],
        "hs_kv_release": [P, I32, P],
        "hs_kv_pool_blocks": [P, ctypes.POINTER(I32), ctypes.POINTER(I32)],
        "hs_handoff_create": [I32, I64, I32, ctypes.c_double, ctypes.POINTER(P)],
        "hs_handoff_free": [P],
        "hs_handoff_push": [P, I32, I32, ctypes.c_double],
        "hs_handoff_pop": [P, ctypes.c_double, P, I32, ctypes.POINTER(I32), ctypes.POINTER(I64),
                           ctypes.POINTER(ctypes.c_double)],
        "hs_handoff_pending": [P, ctypes.POINTER(I32)],
        "hs_stream_read": [P, U64, P, I32, P],
        "hs_decode_step": [P, P, P, P, P, P, P],
        "hs_decode_step_static": [P, P, P, P, P, P, P],
        "hs_model_status": [P, ctypes.POINTER(I32)],
        "hs_kv_lengths": [P, P],
        "hs_kv_sync": [P],
        "hs_kv_write": [P, I32, I32, I32, I32, I32, I32, P, I32],
        "hs_kv_read": [P, I32, I32, I32, I32, I32, I32, P, I32],
        "hs_kv_set_length": [P, I32, I32, I32],
        "hs_replay_kernels": [P, P, I32, I32, P],
        "hs_packed_bytes": [I32, I64, I64, ctypes.POINTER(U64)],
        "hs_pack_matrix": [I32, P, I64, I64, P, P],
        "hs_pack_matrix_heads": [I32, P, I64, I64, I32, P, P],
    }
    for name, args in sig.items():
        fn = getattr(L, name)
        fn.argtypes = args
        fn.restype = ctypes.c_int
    _lib = L
    return L


def check(func: str, rc: int) -> None:
    if rc != HS_OK:
        raise HsError(func, rc, lib().hs_last_error().decode())


def _call(func: str, *args) -> None:
    check(func, getattr(lib(), func)(*args))


def make_config(cfg: dict) -> hs_config:
    c = hs_config()
    for k in ("n_layers", "d_model", "n_heads", "n_kv_heads", "head_dim", "ffn_dim", "vocab", "rope_kind",
              "qkv_bias"):
        setattr(c, k, int(cfg[k]))
    c.rope_theta = float(cfg["rope_theta"])
    c.rms_eps = float(cfg["rms_eps"])
    c.mrope_section[:] = [int(v) for v in cfg["mrope_section"]]
    c.dtype = {"f32": HS_F32, "f16": HS_F16, "bf16": HS_BF16}[cfg["dtype"]]
    return c


def hs_kv_bytes(cfg: dict, n_v: int, s_text: int) -> tuple:
    kv, emb = ctypes.c_uint64(), ctypes.c_uint64()
    _call("hs_kv_bytes", ctypes.byref(make_config(cfg)), n_v, s_text, ctypes.byref(kv), ctypes.byref(emb))
    return kv.value, emb.value


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def stream_read(buf, sink, blocks: int) -> None:
    """Plain streaming read of a device tensor (measurement)."""
    _call("hs_stream_read", _ptr(buf), buf.numel() * buf.element_size(), _ptr(sink), blocks, _stream())


def _stream():
    import torch
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


_DT = {"f32": HS_F32, "f16": HS_F16, "bf16": HS_BF16}


def _is_packed(name: str) -> bool:
    return name.split(".")[-1] in PACKED


def hs_packed_bytes(dtype: str, rows: int, cols: int) -> int:
    out = ctypes.c_uint64()
    _call("hs_packed_bytes", _DT[dtype], rows, cols, ctypes.byref(out))
    return out.value


def pack_matrix(t, dtype: str, head_dim: int = 0):
    """Packed copy (uint8 device tensor) of a row-major [rows, cols] device
    matrix, written on the current stream by hs_pack_matrix, or with head_dim
    by hs_pack_matrix_heads (the q/k/v projections)."""
    import torch
    assert t.is_cuda and t.dim() == 2 and t.is_contiguous()
    rows, cols = t.shape
    out = torch.empty(hs_packed_bytes(dtype, rows, cols), dtype=torch.uint8, device=t.device)
    if head_dim:
        _call("hs_pack_matrix_heads", _DT[dtype], _ptr(t), rows, cols, head_dim, _ptr(out), _stream())
    else:
        _call("hs_pack_matrix", _DT[dtype], _ptr(t), rows, cols, _ptr(out), _stream())
    return out


HEAD_PAIRED = ("wq", "wk", "wv")


def pack_weight(cfg: dict, name: str, t):
    """The tensor the model takes for weight `name`: projection matrices
    packed (q/k/v head-paired), everything else as it is."""
    leaf = name.split(".")[-1]
    if leaf not in PACKED:
        return t
    return pack_matrix(t, cfg["dtype"], cfg["head_dim"] if leaf in HEAD_PAIRED else 0)


def pack_weights(cfg: dict, weights: dict, free_source: bool = False) -> dict:
    """Returns the weight dict with every projection matrix packed; vectors
    and the embedding table pass through.  With free_source the row-major
    matrices are removed from `weights` as they are packed."""
    out = {}
    for name in list(weights):
        out[name] = pack_weight(cfg, name, weights[name])
        if free_source and _is_packed(name):
            del weights[name]
    return out


class Model:
    """A model over device weight tensors named as in the workload generator
    (embed, layers.{i}.wq, ..., final_norm, lm_head).  Row-major projection
    matrices are packed on construction unless packed=True says they already
    are."""

    def __init__(self, cfg: dict, weights: dict, max_batch: int, max_ctx: int, packed: bool = False):
        self.cfg = cfg
        if not packed:
            weights = pack_weights(cfg, weights)
        self._w = weights  # keeps the tensors alive
        L = cfg["n_layers"]
        self._layers = (hs_layer_weights * L)()
        for i in range(L):
            p = f"layers.{i}."
            for n in ("attn_norm", "wq", "wk", "wv", "wo", "mlp_norm", "w_gate", "w_up", "w_down"):
                setattr(self._layers[i], n, weights[p + n].data_ptr())
            if cfg["qkv_bias"]:
                for n in ("bq", "bk", "bv"):
                    setattr(self._layers[i], n, weights[p + n].data_ptr())
        hw = hs_weights()
        hw.embed = weights["embed"].data_ptr()
        if cfg.get("lm_head", True):
            hw.final_norm = weights["final_norm"].data_ptr()
            hw.lm_head = weights["lm_head"].data_ptr()
        hw.layers = self._layers
        self._hw = hw
        self._cfg_c = make_config(cfg)
        h = ctypes.c_void_p()
        _call("hs_model_create", ctypes.byref(self._cfg_c), ctypes.byref(hw), max_batch, max_ctx, ctypes.byref(h))
        self.handle = h
        self.max_batch, self.max_ctx = max_batch, max_ctx

    def reserve_rows(self, rows: int) -> None:
        """Room for `rows` packed prefill rows per pass (grows only)."""
        _call("hs_model_reserve_rows", self.handle, rows)

    def status(self) -> int:
        f = ctypes.c_int32()
        _call("hs_model_status", self.handle, ctypes.byref(f))
        return f.value

    def close(self) -> None:
        if self.handle:
            _call("hs_model_free", self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class KVCache:
    """Per-request contiguous KV cache over a caller-owned uint8 device tensor."""

    def __init__(self, model: Model, n_v, capacity, buf=None):
        import torch
        self.model = model
        self.batch = len(capacity)
        self.n_v = [int(v) for v in n_v]
        self.capacity = [int(c) for c in capacity]
        cfg = model.cfg
        need = sum(hs_kv_bytes(cfg, 0, c)[0] for c in self.capacity)
        if buf is None:
            buf = torch.empty(need, dtype=torch.uint8, device="cuda")
        self.buf = buf
        nv = (ctypes.c_int32 * self.batch)(*self.n_v)
        cap = (ctypes.c_int32 * self.batch)(*self.capacity)
        h = ctypes.c_void_p()
        _call("hs_kv_alloc", model.handle, self.batch, nv, cap, _ptr(buf), buf.numel() * buf.element_size(),
              ctypes.byref(h))
        self.handle = h

    def prefill(self, req: int, emb, text_ids, pos_thw=None, last_logits=None, first_token=None):
        import torch
        if first_token is None:
            first_token = torch.empty(1, dtype=torch.int32, device="cuda")
        _call("hs_prefill_embeddings", self.model.handle, self.handle, req, _ptr(emb), _ptr(text_ids),
              0 if text_ids is None else text_ids.numel(), _ptr(pos_thw), _ptr(last_logits), _ptr(first_token),
              _stream())
        return first_token

    def prefill_batch(self, reqs, emb, text_ids, s_text, pos_thw=None, last_logits=None, first_tokens=None):
        """Prefill of several requests with their rows packed request by
        request: emb holds their vision rows back to back, text_ids their
        text ids, pos_thw (M-RoPE) [3][rows]; returns first_tokens [n]."""
        import torch
        n = len(reqs)
        if first_tokens is None:
            first_tokens = torch.empty(n, dtype=torch.int32, device="cuda")
        r = (ctypes.c_int32 * n)(*reqs)
        t = (ctypes.c_int32 * n)(*s_text)
        _call("hs_prefill_batch", self.model.handle, self.handle, n, r, _ptr(emb), _ptr(text_ids), t, _ptr(pos_thw),
              _ptr(last_logits), _ptr(first_tokens), _stream())
        return first_tokens

    def decode(self, tokens_in, tokens_out, logits=None, hidden_out=None, model=None) -> None:
        """One greedy step; `model` (default: the handle's) may be any model of the same configuration."""
        _call("hs_decode_step", (model or self.model).handle, self.handle, _ptr(tokens_in), _ptr(tokens_out),
              _ptr(logits), _ptr(hidden_out), _stream())

    def decode_static(self, tokens_in, tokens_out, logits=None, hidden_out=None, model=None) -> None:
        """The same step with its scratch in the library's static device array
        (hs_decode_step_static: allocates nothing)."""
        _call("hs_decode_step_static", (model or self.model).handle, self.handle, _ptr(tokens_in), _ptr(tokens_out),
              _ptr(logits), _ptr(hidden_out), _stream())

    def sync(self) -> None:
        """Host mirrors of the lengths from the device (after graph replays)."""
        _call("hs_kv_sync", self.handle)

    def lengths(self) -> list:
        out = (ctypes.c_int32 * self.batch)()
        _call("hs_kv_lengths", self.handle, out)
        return list(out)

    def write(self, req: int, layer: int, kv_sel: int, head: int, pos0: int, rows) -> None:
        n = rows.shape[0]
        _call("hs_kv_write", self.handle, req, layer, kv_sel, head, pos0, n, _ptr(rows), int(rows.is_cuda))

    def read(self, req: int, layer: int, kv_sel: int, head: int, pos0: int, n: int, out) -> None:
        _call("hs_kv_read", self.handle, req, layer, kv_sel, head, pos0, n, _ptr(out), int(out.is_cuda))

    def replay(self, kind: str, count: int, model: "Model | None" = None) -> None:
        """Launches `count` kernels of one kind back to back (measurement)."""
        _call("hs_replay_kernels", (model or self.model).handle, self.handle, HS_K_NAMES.index(kind), count, _stream())

    def set_length(self, req: int, length: int, rope_pos: int) -> None:
        _call("hs_kv_set_length", self.handle, req, length, rope_pos)

    def close(self) -> None:
        if self.handle:
            _call("hs_kv_free", self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class KVPool(KVCache):
    """Block-granular KV cache: `slots` request slots over n_blocks blocks of
    block_tokens positions in a caller-owned (or fresh) uint8 device tensor.
    Requests are admitted into empty slots, prefilled and decoded like
    KVCache requests (slot = request number) and released when done."""

    def __init__(self, model: Model, slots: int, block_tokens: int, n_blocks: int, buf=None):
        import torch
        self.model = model
        self.batch = slots
        self.block_tokens = block_tokens
        block_bytes = hs_kv_bytes(model.cfg, 0, block_tokens)[0]
        if buf is None:
            buf = torch.empty(n_blocks * block_bytes, dtype=torch.uint8, device="cuda")
        self.buf = buf
        h = ctypes.c_void_p()
        _call("hs_kv_pool_create", model.handle, slots, block_tokens, _ptr(buf), buf.numel() * buf.element_size(),
              ctypes.byref(h))
        self.handle = h

    def admit(self, slot: int, n_v: int, capacity: int) -> None:
        _call("hs_kv_admit", self.handle, slot, n_v, capacity, _stream())

    def release(self, slot: int) -> None:
        _call("hs_kv_release", self.handle, slot, _stream())

    def blocks(self) -> tuple:
        """(free, total) blocks."""
        f, n = ctypes.c_int32(), ctypes.c_int32()
        _call("hs_kv_pool_blocks", self.handle, ctypes.byref(f), ctypes.byref(n))
        return f.value, n.value


class Handoff:
    """Aligned batch handoff: requests whose embeddings have arrived wait in
    arrival order until a batch of `align` requests (or the row budget, or
    the oldest request's timeout) is due for prefill."""

    def __init__(self, align: int = 32, max_rows: int = 0, max_pending: int = 4096, timeout_ms: float = 500.0):
        self.align = align
        h = ctypes.c_void_p()
        _call("hs_handoff_create", align, max_rows, max_pending, timeout_ms, ctypes.byref(h))
        self.handle = h

    def push(self, req: int, rows: int, now_ms: float) -> None:
        _call("hs_handoff_push", self.handle, req, rows, now_ms)

    def pop(self, now_ms: float):
        """(requests of the due batch or [], their rows, ms until the next timeout or -1)."""
        out = (ctypes.c_int32 * self.align)()
        n, rows, wait = ctypes.c_int32(), ctypes.c_int64(), ctypes.c_double()
        _call("hs_handoff_pop", self.handle, now_ms, out, self.align, ctypes.byref(n), ctypes.byref(rows),
              ctypes.byref(wait))
        return list(out[:n.value]), rows.value, wait.value

    def pending(self) -> int:
        n = ctypes.c_int32()
        _call("hs_handoff_pending", self.handle, ctypes.byref(n))
        return n.value

    def close(self) -> None:
        if self.handle:
            _call("hs_handoff_free", self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
