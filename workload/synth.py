"""Seeded synthetic inputs shared by the HIP path and the oracle.

This module holds no arithmetic of the method.  It produces weights, vision
embedding rows, token ids, M-RoPE position ids and KV-cache contents from a
counter-based generator, so every tensor is a pure function of
(seed, tensor name, element index) and can be produced on the CPU or on a GPU
with bit-identical results:

* hash: SplitMix64 (Steele, Lea and Flood, "Fast splittable pseudorandom
  number generators", OOPSLA 2014) applied to ``key + (i + 1) * 0x9E3779B97F4A7C15``;
  each 64-bit output supplies four 16-bit fields;
* normal values: a 16-bit field indexes a table of 65,536 standard-normal
  quantiles Phi^-1((j + 0.5) / 65536) (fp32), scaled by an fp32 standard
  deviation and rounded to the storage dtype (round to nearest even);
* uniform integers: the high 32 bits of the hash, multiplied by the range
  width and shifted right by 32.

All integer arithmetic is int64 with wrap-around, all float arithmetic is a
single IEEE fp32 multiply or add, so CPU and GPU agree bit for bit.
"""
from __future__ import annotations

import statistics
from typing import Sequence

import numpy as np
import torch

MASK64 = (1 << 64) - 1
GAMMA = 0x9E3779B97F4A7C15
MIX1 = 0xBF58476D1CE4E5B9
MIX2 = 0x94D049BB133111EB


def _s64(u: int) -> int:
    """uint64 bit pattern -> int64 value with the same bits."""
    u &= MASK64
    return u - (1 << 64) if u >= (1 << 63) else u


def splitmix64_py(z: int) -> int:
    """Reference SplitMix64 finaliser on Python ints (uint64 semantics)."""
    z &= MASK64
    z = ((z ^ (z >> 30)) * MIX1) & MASK64
    z = ((z ^ (z >> 27)) * MIX2) & MASK64
    return z ^ (z >> 31)


def fnv1a64(text: str) -> int:
    h = 0xCBF29CE484222325
    for byte in text.encode():
        h ^= byte
        h = (h * 0x100000001B3) & MASK64
    return h


def tensor_key(seed: int, name: str) -> int:
    """uint64 key of one named tensor under one seed."""
    return splitmix64_py(fnv1a64(name) ^ ((seed * GAMMA) & MASK64))


def _lsr(z: torch.Tensor, s: int) -> torch.Tensor:
    """Logical right shift of int64 bit patterns."""
    return (z >> s) & ((1 << (64 - s)) - 1)


def hash_stream(key: int, start: int, count: int, device) -> torch.Tensor:
    """SplitMix64 outputs start..start+count-1 of the stream with this key, as
    int64 bit patterns."""
    i = torch.arange(start + 1, start + count + 1, dtype=torch.int64, device=device)
    z = i * _s64(GAMMA) + _s64(key)
    z = z ^ _lsr(z, 30)
    z = z * _s64(MIX1)
    z = z ^ _lsr(z, 27)
    z = z * _s64(MIX2)
    z = z ^ _lsr(z, 31)
    return z


_QTABLE: dict = {}


def normal_quantile_table(device) -> torch.Tensor:
    key = str(device)
    if key not in _QTABLE:
        nd = statistics.NormalDist()
        q = np.array([nd.inv_cdf((j + 0.5) / 65536.0) for j in range(65536)], dtype=np.float32)
        _QTABLE[key] = torch.from_numpy(q).to(device)
    return _QTABLE[key]


_DTYPES = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}

CHUNK_HASHES = 1 << 22


def _fields16(key: int, start_elem: int, n: int, device) -> torch.Tensor:
    """16-bit fields for elements start_elem .. start_elem+n-1 (start_elem % 4 == 0)."""
    assert start_elem % 4 == 0
    nh = (n + 3) // 4
    z = hash_stream(key, start_elem // 4, nh, device)
    # field f of hash h is bits 16f..16f+15 (an arithmetic shift followed by
    # the 16-bit mask yields the same bits as a logical one)
    shifts = torch.tensor([0, 16, 32, 48], dtype=torch.int64, device=device)
    f = (z.unsqueeze(1) >> shifts) & 0xFFFF
    return f.reshape(-1)[:n]


def normal(seed: int, name: str, shape: Sequence[int], std: float, dtype: str, device="cpu",
           mean: float | None = None) -> torch.Tensor:
    """~N(mean, std^2) values in the storage dtype (mean None -> 0)."""
    n = int(np.prod(shape)) if len(shape) else 1
    out = torch.empty(n, dtype=_DTYPES[dtype], device=device)
    table = normal_quantile_table(device)
    key = tensor_key(seed, name)
    std_t = torch.tensor(std, dtype=torch.float32, device=device)
    mean_t = None if mean is None else torch.tensor(mean, dtype=torch.float32, device=device)
    step = CHUNK_HASHES * 4
    for s in range(0, n, step):
        m = min(step, n - s)
        v = table[_fields16(key, s, m, device)] * std_t
        if mean_t is not None:
            v = mean_t + v
        out[s:s + m] = v.to(out.dtype)
    return out.reshape(tuple(shape))


def uniform_int(seed: int, name: str, n: int, lo: int, hi: int, device="cpu") -> torch.Tensor:
    """n integers uniform in [lo, hi] inclusive, int32."""
    assert hi >= lo and hi - lo + 1 < (1 << 31)
    width = hi - lo + 1
    z = hash_stream(tensor_key(seed, name), 0, n, device)
    u = _lsr(z, 32)
    return (lo + ((u * width) >> 32)).to(torch.int32)


# --------------------------------------------------------------------------
# Workload recipes
# --------------------------------------------------------------------------

def weight_names(cfg: dict) -> list:
    names = ["embed"]
    for layer in range(cfg["n_layers"]):
        p = f"layers.{layer}."
        names += [p + n for n in ("attn_norm", "wq", "wk", "wv", "wo", "mlp_norm", "w_gate", "w_up", "w_down")]
        if cfg["qkv_bias"]:
            names += [p + "bq", p + "bk", p + "bv"]
    if cfg.get("lm_head", True):
        names += ["final_norm", "lm_head"]
    return names


def weight_shape(cfg: dict, name: str) -> tuple:
    d, nh, nkv, hd, F, V = (cfg[k] for k in ("d_model", "n_heads", "n_kv_heads", "head_dim", "ffn_dim", "vocab"))
    base = name.split(".")[-1]
    return {
        "embed": (V, d), "lm_head": (V, d), "final_norm": (d,), "attn_norm": (d,), "mlp_norm": (d,),
        "wq": (nh * hd, d), "wk": (nkv * hd, d), "wv": (nkv * hd, d), "wo": (d, nh * hd),
        "bq": (nh * hd,), "bk": (nkv * hd,), "bv": (nkv * hd,),
        "w_gate": (F, d), "w_up": (F, d), "w_down": (d, F),
    }[base]


def make_weight(cfg: dict, name: str, device="cpu", seed: int | None = None) -> torch.Tensor:
    """Linear and embedding weights ~N(0, 0.02); norm gains 1 + N(0, 0.02);
    biases ~N(0, 0.02)."""
    seed = cfg["seed"] if seed is None else seed
    shape = weight_shape(cfg, name)
    if name.endswith("norm"):
        return normal(seed, name, shape, 0.02, cfg["dtype"], device, mean=1.0)
    return normal(seed, name, shape, 0.02, cfg["dtype"], device)


def make_weights(cfg: dict, device="cpu", seed: int | None = None) -> dict:
    return {n: make_weight(cfg, n, device, seed) for n in weight_names(cfg)}


def request_lengths(cfg: dict) -> tuple:
    """(n_v[B], s_text[B]) as Python lists, per the workload's length mix."""
    B, seed = cfg["batch"], cfg["seed"]
    nv, st = cfg["n_v"], cfg["s_text"]
    n_v = ([int(nv)] * B if isinstance(nv, int)
           else uniform_int(seed, "n_v", B, nv[0], nv[1]).tolist())
    s_text = ([int(st)] * B if isinstance(st, int)
              else uniform_int(seed, "s_text", B, st[0], st[1]).tolist())
    return n_v, s_text


def vision_rows(cfg: dict, req: int, n_v: int, device="cpu") -> torch.Tensor:
    """Projected vision embedding [n_v, d] ~N(0, 1)."""
    return normal(cfg["seed"], f"req.{req}.vision", (n_v, cfg["d_model"]), 1.0, cfg["dtype"], device)


def text_ids(cfg: dict, req: int, s_text: int, device="cpu") -> torch.Tensor:
    return uniform_int(cfg["seed"], f"req.{req}.text", s_text, 0, cfg["vocab"] - 1, device)


def mrope_positions(n_v: int, s_text: int) -> torch.Tensor:
    """(t, h, w) position ids [3, n_v + s_text] int32: vision row i sits at
    t = 0, h = i // W, w = i % W with W = ceil(sqrt(n_v)); text token j at
    t = h = w = (largest vision id) + 1 + j."""
    W = max(1, int(np.ceil(np.sqrt(n_v)))) if n_v > 0 else 1
    i = np.arange(n_v)
    vis = np.stack([np.zeros(n_v, dtype=np.int64), i // W, i % W]) if n_v > 0 else np.zeros((3, 0), np.int64)
    start = int(vis.max()) + 1 if n_v > 0 else 0
    txt = np.tile(start + np.arange(s_text), (3, 1))
    return torch.from_numpy(np.concatenate([vis, txt], axis=1).astype(np.int32))


def kv_lengths(cfg: dict) -> list:
    lo, hi = cfg["kv_len"]
    return uniform_int(cfg["seed"], "kv_len", cfg["batch"], lo, hi).tolist()


def kv_block(cfg: dict, req: int, layer: int, kv_sel: int, head: int, n: int, device="cpu") -> torch.Tensor:
    """Synthetic cache rows [n, d_h] ~N(0, 1) for one (request, layer, K|V, head)."""
    return normal(cfg["seed"], f"req.{req}.kv.{layer}.{kv_sel}.{head}", (n, cfg["head_dim"]), 1.0,
                  cfg["dtype"], device)


def decode_tokens(cfg: dict, req: int, n: int, device="cpu") -> torch.Tensor:
    """Token ids fed to teacher-forced decode steps."""
    return uniform_int(cfg["seed"], f"req.{req}.decode", n, 0, cfg["vocab"] - 1, device)
