"""ctypes wrapper of the plain C oracle (hs_oracle.c).

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the benchmark's
CPU-baseline leg may use this module; the product path never does.  It imports
nothing from the HIP package.

Tensors handed to the oracle are CPU torch tensors (contiguous) in the storage
dtype; the wrapper keeps references so the C side can hold raw pointers.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np
import torch

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "hs_oracle.c")
LIB = os.path.join(HERE, "liboracle.so")

F32, F16, BF16 = 0, 1, 2
DTYPE_CODE = {"f32": F32, "f16": F16, "bf16": BF16}
TORCH_DTYPE = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}


def build(force: bool = False) -> str:
    """Compile the oracle with gcc: single-threaded, no fast-math, no FMA
    contraction."""
    if force or not os.path.exists(LIB) or os.path.getmtime(LIB) < max(
            os.path.getmtime(SRC), os.path.getmtime(os.path.join(HERE, "hs_oracle.h"))):
        tmp = LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-Wall", "-ffp-contract=off", "-fno-fast-math", "-fPIC",
                               "-shared", "-o", tmp, SRC, "-lm"])
        os.replace(tmp, LIB)
    return LIB


class OrConfig(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32), ("n_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("ffn_dim", ctypes.c_int32),
                ("vocab", ctypes.c_int32), ("rope_theta", ctypes.c_float), ("rms_eps", ctypes.c_float),
                ("rope_kind", ctypes.c_int32), ("mrope_section", ctypes.c_int32 * 3),
                ("qkv_bias", ctypes.c_int32), ("dtype", ctypes.c_int32)]


class OrLayer(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("attn_norm", "wq", "wk", "wv", "bq", "bk", "bv", "wo", "mlp_norm",
                                                 "w_gate", "w_up", "w_down")]


class OrModel(ctypes.Structure):
    _fields_ = [("cfg", OrConfig), ("embed", ctypes.c_void_p), ("final_norm", ctypes.c_void_p),
                ("lm_head", ctypes.c_void_p), ("layers", ctypes.POINTER(OrLayer))]


class OrSeq(ctypes.Structure):
    _fields_ = [("cap", ctypes.c_int32), ("len", ctypes.c_int32), ("rope_pos", ctypes.c_int32),
                ("kv", ctypes.POINTER(ctypes.c_float))]


_lib = None


def lib():
    global _lib
    if _lib is None:
        _lib = ctypes.CDLL(build())
        P, I32, I64, F = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float
        _lib.or_transfer_bytes.argtypes = [ctypes.POINTER(OrConfig), I64, I64, ctypes.POINTER(ctypes.c_uint64),
                                           ctypes.POINTER(ctypes.c_uint64)]
        _lib.or_round.argtypes = [I32, F]
        _lib.or_round.restype = F
        _lib.or_f32_to_f16_bits.argtypes = [F]
        _lib.or_f32_to_f16_bits.restype = ctypes.c_uint16
        _lib.or_f32_to_bf16_bits.argtypes = [F]
        _lib.or_f32_to_bf16_bits.restype = ctypes.c_uint16
        _lib.or_rmsnorm.argtypes = [I32, P, P, I32, F, P]
        _lib.or_rope_cos_sin.argtypes = [F, I32, I32, I32, ctypes.POINTER(F), ctypes.POINTER(F)]
        _lib.or_rope_rotate.argtypes = [ctypes.POINTER(OrConfig), P, P]
        _lib.or_attention.argtypes = [I32, I32, P, P, I64, P, I64, P]
        _lib.or_silu.argtypes = [F]
        _lib.or_silu.restype = F
        _lib.or_argmax.argtypes = [I32, P]
        _lib.or_argmax.restype = I32
        _lib.or_seq_init.argtypes = [ctypes.POINTER(OrModel), ctypes.POINTER(OrSeq), I32]
        _lib.or_seq_free.argtypes = [ctypes.POINTER(OrSeq)]
        _lib.or_seq_write_kv.argtypes = [ctypes.POINTER(OrModel), ctypes.POINTER(OrSeq), I32, I32, I32, I32, I32, P]
        _lib.or_seq_read_kv.argtypes = [ctypes.POINTER(OrModel), ctypes.POINTER(OrSeq), I32, I32, I32, I32, I32, P]
        _lib.or_seq_set_len.argtypes = [ctypes.POINTER(OrSeq), I32, I32]
        _lib.or_forward_row.argtypes = [ctypes.POINTER(OrModel), ctypes.POINTER(OrSeq), P, P, P, P]
        _lib.or_prefill.argtypes = [ctypes.POINTER(OrModel), ctypes.POINTER(OrSeq), P, I32, P, I32, P, P, P]
        _lib.or_decode.argtypes = [ctypes.POINTER(OrModel), ctypes.POINTER(OrSeq), I32, P, P, P]
    return _lib


def make_config(cfg: dict) -> OrConfig:
    c = OrConfig()
    for k in ("n_layers", "d_model", "n_heads", "n_kv_heads", "head_dim", "ffn_dim", "vocab", "rope_kind",
              "qkv_bias"):
        setattr(c, k, int(cfg[k]))
    c.rope_theta = float(cfg["rope_theta"])
    c.rms_eps = float(cfg["rms_eps"])
    c.mrope_section[:] = [int(v) for v in cfg["mrope_section"]]
    c.dtype = DTYPE_CODE[cfg["dtype"]]
    return c


def _ptr(t: torch.Tensor | None):
    if t is None:
        return None
    assert t.device.type == "cpu" and t.is_contiguous()
    return ctypes.c_void_p(t.data_ptr())


def _f32(a) -> torch.Tensor:
    return torch.as_tensor(a, dtype=torch.float32).contiguous()


# ---------------------------------------------------------------------------
# building blocks
# ---------------------------------------------------------------------------

def transfer_bytes(cfg: dict, n_v: int, s_text: int) -> tuple:
    kv, emb = ctypes.c_uint64(), ctypes.c_uint64()
    rc = lib().or_transfer_bytes(ctypes.byref(make_config(cfg)), n_v, s_text, ctypes.byref(kv), ctypes.byref(emb))
    if rc != 0:
        raise ValueError(f"or_transfer_bytes rc={rc}")
    return kv.value, emb.value


def round_to(dtype: str, x) -> np.ndarray:
    code = DTYPE_CODE[dtype]
    return np.array([lib().or_round(code, float(v)) for v in np.asarray(x, dtype=np.float32).ravel()],
                    dtype=np.float32).reshape(np.shape(x))


def f16_bits(x: float) -> int:
    return int(lib().or_f32_to_f16_bits(float(x)))


def bf16_bits(x: float) -> int:
    return int(lib().or_f32_to_bf16_bits(float(x)))


def rmsnorm(x, gain: torch.Tensor, dtype: str, eps: float) -> np.ndarray:
    x = _f32(x)
    out = torch.empty_like(x)
    lib().or_rmsnorm(x.numel(), _ptr(x), _ptr(gain.contiguous()), DTYPE_CODE[dtype], eps, _ptr(out))
    return out.numpy()


def rope_cos_sin(theta: float, head_dim: int, pair: int, pos: int) -> tuple:
    c, s = ctypes.c_float(), ctypes.c_float()
    lib().or_rope_cos_sin(theta, head_dim, pair, pos, ctypes.byref(c), ctypes.byref(s))
    return c.value, s.value


def rope_rotate(cfg: dict, vec, pos3) -> np.ndarray:
    v = _f32(vec).clone()
    p = torch.tensor(list(pos3), dtype=torch.int32)
    lib().or_rope_rotate(ctypes.byref(make_config(cfg)), _ptr(v), _ptr(p))
    return v.numpy()


def attention(q, k, v) -> np.ndarray:
    q, k, v = _f32(q), _f32(k), _f32(v)
    n_t, d_h = k.shape
    o = torch.empty(d_h, dtype=torch.float32)
    lib().or_attention(n_t, d_h, _ptr(q), _ptr(k), d_h, _ptr(v), d_h, _ptr(o))
    return o.numpy()


def silu(z: float) -> float:
    return float(lib().or_silu(float(z)))


def argmax(v) -> int:
    v = _f32(v)
    return int(lib().or_argmax(v.numel(), _ptr(v)))


# ---------------------------------------------------------------------------
# whole model
# ---------------------------------------------------------------------------

class Model:
    """Oracle model over CPU weight tensors named as in workload.synth."""

    def __init__(self, cfg: dict, weights: dict):
        self.cfg = cfg
        self._keep = {k: v.contiguous() for k, v in weights.items()}
        w = self._keep
        L = cfg["n_layers"]
        self._layers = (OrLayer * L)()
        for i in range(L):
            p = f"layers.{i}."
            lay = self._layers[i]
            for n in ("attn_norm", "wq", "wk", "wv", "wo", "mlp_norm", "w_gate", "w_up", "w_down"):
                setattr(lay, n, w[p + n].data_ptr())
            for n in ("bq", "bk", "bv"):
                setattr(lay, n, w[p + n].data_ptr() if cfg["qkv_bias"] else None)
        self.m = OrModel()
        self.m.cfg = make_config(cfg)
        self.m.embed = w["embed"].data_ptr()
        has_head = cfg.get("lm_head", True)
        self.m.final_norm = w["final_norm"].data_ptr() if has_head else None
        self.m.lm_head = w["lm_head"].data_ptr() if has_head else None
        self.m.layers = self._layers

    def new_seq(self, cap: int) -> "Seq":
        return Seq(self, cap)


class Seq:
    def __init__(self, model: Model, cap: int):
        self.model = model
        self.s = OrSeq()
        rc = lib().or_seq_init(ctypes.byref(model.m), ctypes.byref(self.s), cap)
        if rc != 0:
            raise ValueError(f"or_seq_init rc={rc}")

    def __del__(self):
        try:
            lib().or_seq_free(ctypes.byref(self.s))
        except Exception:
            pass

    @property
    def len(self) -> int:
        return self.s.len

    @property
    def rope_pos(self) -> int:
        return self.s.rope_pos

    def prefill(self, emb: torch.Tensor | None, text_ids, pos_thw=None):
        cfg = self.model.cfg
        n_v = 0 if emb is None else emb.shape[0]
        ids = torch.as_tensor(text_ids, dtype=torch.int32).contiguous()
        pos = None if pos_thw is None else torch.as_tensor(pos_thw, dtype=torch.int32).contiguous()
        logits = torch.empty(cfg["vocab"], dtype=torch.float32) if cfg.get("lm_head", True) else None
        tok = ctypes.c_int32(-1)
        rc = lib().or_prefill(ctypes.byref(self.model.m), ctypes.byref(self.s),
                              _ptr(None if emb is None else emb.contiguous()), n_v, _ptr(ids), ids.numel(),
                              _ptr(pos), _ptr(logits), ctypes.byref(tok))
        if rc != 0:
            raise ValueError(f"or_prefill rc={rc}")
        return (None if logits is None else logits.numpy()), tok.value

    def decode(self, token: int):
        cfg = self.model.cfg
        logits = torch.empty(cfg["vocab"], dtype=torch.float32) if cfg.get("lm_head", True) else None
        hidden = torch.empty(cfg["d_model"], dtype=torch.float32)
        tok = ctypes.c_int32(-1)
        rc = lib().or_decode(ctypes.byref(self.model.m), ctypes.byref(self.s), int(token), _ptr(logits),
                             _ptr(hidden), ctypes.byref(tok))
        if rc != 0:
            raise ValueError(f"or_decode rc={rc}")
        return (None if logits is None else logits.numpy()), hidden.numpy(), tok.value

    def forward_row(self, x, pos3, want_logits: bool = True):
        cfg = self.model.cfg
        x = _f32(x)
        p = torch.tensor(list(pos3), dtype=torch.int32)
        logits = torch.empty(cfg["vocab"], dtype=torch.float32) if want_logits and cfg.get("lm_head", True) else None
        hidden = torch.empty(cfg["d_model"], dtype=torch.float32)
        rc = lib().or_forward_row(ctypes.byref(self.model.m), ctypes.byref(self.s), _ptr(x), _ptr(p), _ptr(hidden),
                                  _ptr(logits))
        if rc != 0:
            raise ValueError(f"or_forward_row rc={rc}")
        return (None if logits is None else logits.numpy()), hidden.numpy()

    def write_kv(self, layer: int, kv_sel: int, head: int, pos0: int, rows) -> None:
        r = _f32(rows)
        rc = lib().or_seq_write_kv(ctypes.byref(self.model.m), ctypes.byref(self.s), layer, kv_sel, head, pos0,
                                   r.shape[0], _ptr(r))
        if rc != 0:
            raise ValueError(f"or_seq_write_kv rc={rc}")

    def read_kv(self, layer: int, kv_sel: int, head: int, pos0: int, n: int) -> np.ndarray:
        out = torch.empty((n, self.model.cfg["head_dim"]), dtype=torch.float32)
        rc = lib().or_seq_read_kv(ctypes.byref(self.model.m), ctypes.byref(self.s), layer, kv_sel, head, pos0, n,
                                  _ptr(out))
        if rc != 0:
            raise ValueError(f"or_seq_read_kv rc={rc}")
        return out.numpy()

    def set_len(self, length: int, rope_pos: int) -> None:
        rc = lib().or_seq_set_len(ctypes.byref(self.s), length, rope_pos)
        if rc != 0:
            raise ValueError(f"or_seq_set_len rc={rc}")
