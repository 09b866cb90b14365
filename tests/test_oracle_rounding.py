"""Pins of the oracle's storage-rounding placement, its K/V cache contents and
its cache copy hooks, against the transformers LLaMA and Qwen2.5-VL text
decoders run in fp64.

The library decoders supply the layer wiring (pre-norm residual blocks, head
split and GQA grouping, q/k/v/o projections, the SwiGLU MLP, the final norm
and head, 3-section M-RoPE).  Hooks put on them the precision that the
oracle's reading prescribes, written out here from that reading and not taken
from the oracle:
  * state (residual stream, projections before rounding, logits) is fp32:
    each is rounded to fp32 where it is produced;
  * R(.) (fp32 value rounded to nearest even into the storage dtype) at h and
    h2 (the two norms' outputs), the final norm's output, q/k/v after RoPE,
    the attention output o and the SwiGLU output a;
  * RMSNorm, the RoPE angles and cos/sin, and softmax are evaluated in fp64
    (the library's own RMSNorm, rotary table and eager softmax run in fp32);
    cos/sin are the fp32 values of fp64 cos/sin of the fp64 angle.
With that, the oracle must agree with the hooked decoder to fp32 rounding of
the logits, bit for bit on the cached K/V rows, and dropping any single
rounding point from the hooks must move the library decoder visibly away from
the oracle, so a dropped or moved R(.) in the oracle fails here.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

from oracle import oracle as O
from workload import synth

STORE = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}
POINTS = ("h", "q", "k", "v", "o", "h2", "a", "final")


def _cfg(**kw):
    base = dict(name="round", n_layers=2, d_model=64, n_heads=4, n_kv_heads=2, head_dim=16, ffn_dim=96, vocab=97,
                rope_theta=1e4, rms_eps=1e-5, rope_kind=0, mrope_section=(0, 0, 0), qkv_bias=0, dtype="f16",
                lm_head=True, seed=23)
    base.update(kw)
    return base


def _rel(a, b):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    return float(np.max(np.abs(a - b)) / np.max(np.abs(b)))


def _fp32(t: torch.Tensor) -> torch.Tensor:
    return t.float().double()


class _Reading:
    """Hooks that give a library decoder (fp64 parameters) the oracle reading's
    precision; `skip` names rounding points left out (fp32 kept)."""

    def __init__(self, cfg: dict, model, text_model, skip=()):
        self.cfg, self.skip = cfg, set(skip)
        self.store = STORE[cfg["dtype"]]
        self.kv = {}  # layer -> (K, V) as the attention saw them, [n_kv, T, d_h]
        self.handles = []
        self.eps = float(np.float32(cfg["rms_eps"]))
        tm = text_model
        tm.rotary_emb.forward = self._rotary
        for i, layer in enumerate(tm.layers):
            layer.self_attn.layer_idx = i
            self._hook_layer(layer)
        self.handles.append(tm.norm.register_forward_pre_hook(self._round_state_in_place))
        self.handles.append(tm.norm.register_forward_hook(self._norm("final")))
        self.model = model

    def R(self, t: torch.Tensor, point: str) -> torch.Tensor:
        t = _fp32(t)
        return t if point in self.skip else t.to(self.store).double()

    # residual stream: rounded to fp32 in place where it enters a norm, so the
    # layer's own `residual` reference (the same tensor) is rounded too
    @staticmethod
    def _round_state_in_place(_mod, args):
        args[0].copy_(_fp32(args[0]))

    def _norm(self, point):
        def hook(mod, args, _out):
            x = args[0]
            rsq = 1.0 / torch.sqrt((x * x).mean(-1, keepdim=True) + self.eps)
            return self.R(x * rsq * mod.weight, point)
        return hook

    def _hook_layer(self, layer):
        at, mlp = layer.self_attn, layer.mlp
        self.handles += [
            layer.input_layernorm.register_forward_pre_hook(self._round_state_in_place),
            layer.input_layernorm.register_forward_hook(self._norm("h")),
            layer.post_attention_layernorm.register_forward_pre_hook(self._round_state_in_place),
            layer.post_attention_layernorm.register_forward_hook(self._norm("h2")),
            at.q_proj.register_forward_hook(lambda m, a, out: _fp32(out)),
            at.k_proj.register_forward_hook(lambda m, a, out: _fp32(out)),
            at.v_proj.register_forward_hook(lambda m, a, out: _fp32(out)),
            mlp.gate_proj.register_forward_hook(lambda m, a, out: _fp32(out)),
            mlp.up_proj.register_forward_hook(lambda m, a, out: _fp32(out)),
            mlp.down_proj.register_forward_pre_hook(lambda m, a: (self.R(a[0], "a"),)),
        ]

    def _rotary(self, x, position_ids):
        """cos/sin of the reading: fp32 values of fp64 cos/sin of pos * theta^(-2i/d_h)."""
        d_h = self.cfg["head_dim"]
        i = np.arange(d_h // 2, dtype=np.float64)
        inv = np.power(np.float64(np.float32(self.cfg["rope_theta"])), -2.0 * i / d_h)
        pos = position_ids.double().numpy()
        ang = pos[..., None] * inv
        cos = np.cos(ang).astype(np.float32).astype(np.float64)
        sin = np.sin(ang).astype(np.float32).astype(np.float64)
        cos, sin = (torch.from_numpy(np.concatenate([t, t], -1)) for t in (cos, sin))
        return cos, sin

    def attention(self, module, q, k, v, mask, scaling, dropout=0.0, **kw):
        """Causal softmax attention in fp64 over the rounded q/k/v; output R(o)."""
        q, k, v = self.R(q, "q"), self.R(k, "k"), self.R(v, "v")
        self.kv[module.layer_idx] = (k[0].clone(), v[0].clone())
        g = q.shape[1] // k.shape[1]
        k = k.repeat_interleave(g, dim=1)  # query head i reads KV head i // g
        v = v.repeat_interleave(g, dim=1)
        T = q.shape[2]
        s = (q @ k.transpose(2, 3)) * (1.0 / np.sqrt(self.cfg["head_dim"]))
        s = s.masked_fill(torch.triu(torch.ones(T, T, dtype=torch.bool), 1), float("-inf"))
        p = torch.softmax(s, dim=-1)
        o = self.R(p @ v, "o")
        return o.transpose(1, 2).contiguous(), None


def _register(reading: _Reading) -> str:
    from transformers import AttentionInterface
    from transformers.masking_utils import ALL_MASK_ATTENTION_FUNCTIONS, sdpa_mask
    name = "oracle_reading"
    AttentionInterface.register(name, lambda *a, **kw: reading.attention(*a, **kw))
    ALL_MASK_ATTENTION_FUNCTIONS.register(name, sdpa_mask)
    return name


def _llama(cfg, W, skip=()):
    from transformers import LlamaConfig, LlamaForCausalLM
    c = LlamaConfig(vocab_size=cfg["vocab"], hidden_size=cfg["d_model"], intermediate_size=cfg["ffn_dim"],
                    num_hidden_layers=cfg["n_layers"], num_attention_heads=cfg["n_heads"],
                    num_key_value_heads=cfg["n_kv_heads"], head_dim=cfg["head_dim"], rms_norm_eps=cfg["rms_eps"],
                    rope_parameters={"rope_type": "default", "rope_theta": cfg["rope_theta"]},
                    tie_word_embeddings=False, attn_implementation="eager", max_position_embeddings=4096,
                    bos_token_id=None, eos_token_id=None, pad_token_id=None)
    m = LlamaForCausalLM(c).double().eval()
    sd = {"model.embed_tokens.weight": W["embed"], "model.norm.weight": W["final_norm"], "lm_head.weight": W["lm_head"]}
    for i in range(cfg["n_layers"]):
        p, q = f"layers.{i}.", f"model.layers.{i}."
        for a, b in (("wq", "self_attn.q_proj.weight"), ("wk", "self_attn.k_proj.weight"),
                     ("wv", "self_attn.v_proj.weight"), ("wo", "self_attn.o_proj.weight"),
                     ("w_gate", "mlp.gate_proj.weight"), ("w_up", "mlp.up_proj.weight"),
                     ("w_down", "mlp.down_proj.weight"), ("attn_norm", "input_layernorm.weight"),
                     ("mlp_norm", "post_attention_layernorm.weight")):
            sd[q + b] = W[p + a]
    m.load_state_dict({k: v.double() for k, v in sd.items()})
    reading = _Reading(cfg, m, m.model, skip)
    m.config._attn_implementation = _register(reading)

    def run(rows, positions):
        with torch.no_grad():
            out = m(inputs_embeds=torch.cat(rows)[None], use_cache=False)
        return out.logits[0, -1].numpy()
    return run, reading


def _qwen(cfg, W, skip=()):
    from transformers.models.qwen2_5_vl.configuration_qwen2_5_vl import Qwen2_5_VLTextConfig
    from transformers.models.qwen2_5_vl.modeling_qwen2_5_vl import Qwen2_5_VLTextModel
    qc = Qwen2_5_VLTextConfig(vocab_size=cfg["vocab"], hidden_size=cfg["d_model"], intermediate_size=cfg["ffn_dim"],
                              num_hidden_layers=cfg["n_layers"], num_attention_heads=cfg["n_heads"],
                              num_key_value_heads=cfg["n_kv_heads"], rms_norm_eps=cfg["rms_eps"],
                              rope_parameters={"rope_type": "default", "rope_theta": cfg["rope_theta"],
                                               "mrope_section": list(cfg["mrope_section"])},
                              attn_implementation="eager", max_position_embeddings=4096,
                              bos_token_id=None, eos_token_id=None, pad_token_id=None)
    m = Qwen2_5_VLTextModel(qc).double().eval()
    sd = {"embed_tokens.weight": W["embed"], "norm.weight": W["final_norm"]}
    for i in range(cfg["n_layers"]):
        p = f"layers.{i}."
        for a, b in (("wq", "self_attn.q_proj.weight"), ("wk", "self_attn.k_proj.weight"),
                     ("wv", "self_attn.v_proj.weight"), ("wo", "self_attn.o_proj.weight"),
                     ("bq", "self_attn.q_proj.bias"), ("bk", "self_attn.k_proj.bias"), ("bv", "self_attn.v_proj.bias"),
                     ("w_gate", "mlp.gate_proj.weight"), ("w_up", "mlp.up_proj.weight"),
                     ("w_down", "mlp.down_proj.weight"), ("attn_norm", "input_layernorm.weight"),
                     ("mlp_norm", "post_attention_layernorm.weight")):
            sd[p + b] = W[p + a]
    m.load_state_dict({k: v.double() for k, v in sd.items()})
    reading = _Reading(cfg, m, m, skip)
    m.config._attn_implementation = _register(reading)
    lm = W["lm_head"].double()

    def run(rows, positions):
        with torch.no_grad():
            h = m(inputs_embeds=torch.cat(rows)[None], position_ids=positions[:, None, :].long(),
                  use_cache=False).last_hidden_state[0, -1]
        return _fp32(lm @ h).numpy()
    return run, reading


CASES = {
    "llama_f16": dict(dtype="f16"),
    "llama_bf16": dict(dtype="bf16"),
    "llama_f32": dict(dtype="f32"),
    "qwen_bf16": dict(dtype="bf16", rope_theta=1e6, rms_eps=1e-6, rope_kind=1, mrope_section=(2, 3, 3), qkv_bias=1),
}


def _run_case(case: str, skip=(), n_dec: int = 2):
    """Oracle and hooked library decoder over prefill + n_dec greedy steps.
    Returns the largest relative logit gap, the oracle sequence, the last
    hooked run's captured K/V and the oracle tokens."""
    cfg = _cfg(**CASES[case])
    W = synth.make_weights(cfg)
    n_v, s_text = 6, 4
    emb = synth.vision_rows(cfg, 0, n_v)
    ids = synth.text_ids(cfg, 0, s_text)
    qwen = cfg["rope_kind"] == 1
    pos = synth.mrope_positions(n_v, s_text) if qwen else torch.arange(n_v + s_text, dtype=torch.int32)[None].repeat(3, 1)
    seq = O.Model(cfg, W).new_seq(n_v + s_text + n_dec)
    logits, tok = seq.prefill(emb, ids, pos if qwen else None)
    run, reading = (_qwen if qwen else _llama)(cfg, W, skip)
    rows = [emb.double(), W["embed"].double()[ids.long()]]
    worst = _rel(logits, run(rows, pos))
    toks = [tok]
    for _ in range(n_dec):
        p = seq.rope_pos
        logits, _, tok = seq.decode(toks[-1])
        rows.append(W["embed"].double()[toks[-1]][None])
        pos = torch.cat([pos, torch.full((3, 1), p, dtype=torch.int32)], 1)
        worst = max(worst, _rel(logits, run(rows, pos)))
        toks.append(tok)
    for h in reading.handles:
        h.remove()
    return worst, seq, reading.kv, cfg


@pytest.mark.parametrize("case", list(CASES))
def test_oracle_matches_library_decoder_with_reading_precision(case):
    """Logits to fp32 rounding, and every cached K/V row (each layer, KV head
    and position: the oracle's read_kv) bit-equal to the K/V rows the hooked
    library attention saw."""
    worst, seq, kv, cfg = _run_case(case)
    assert worst <= 1e-6, worst
    T = seq.len
    for layer in range(cfg["n_layers"]):
        K, V = kv[layer]
        assert K.shape[1] == T
        for head in range(cfg["n_kv_heads"]):
            for sel, ref in ((0, K), (1, V)):
                got = seq.read_kv(layer, sel, head, 0, T)
                assert np.array_equal(got.astype(np.float64), ref[head].numpy()), (layer, head, sel)


@pytest.mark.parametrize("point", POINTS)
@pytest.mark.parametrize("case", ["llama_f16", "qwen_bf16"])
def test_each_rounding_point_is_visible(case, point):
    """Leaving one R(.) out of the hooked decoder moves it far from the oracle,
    so the test above would catch an oracle that dropped or moved it."""
    exact, _, _, _ = _run_case(case, n_dec=1)
    dropped, _, _, _ = _run_case(case, skip=(point,), n_dec=1)
    assert dropped > 1e-5 and dropped > 30 * exact, (point, dropped, exact)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("rope_kind", [0, 1])
def test_cache_copy_hooks_reproduce_the_prefilled_sequence(dtype, rope_kind):
    """read_kv of every row of a prefilled sequence, write_kv of those rows
    into a fresh sequence and set_len(len, next RoPE position) give a
    sequence whose next decode step is bit-equal to the original's; with a
    wrong RoPE position or a missing row it is not."""
    kw = dict(dtype=dtype)
    if rope_kind:
        kw.update(rope_theta=1e6, rms_eps=1e-6, rope_kind=1, mrope_section=(2, 3, 3), qkv_bias=1)
    cfg = _cfg(**kw)
    W = synth.make_weights(cfg)
    om = O.Model(cfg, W)
    n_v, s_text = 9, 3
    emb = synth.vision_rows(cfg, 1, n_v)
    ids = synth.text_ids(cfg, 1, s_text)
    pos = synth.mrope_positions(n_v, s_text) if rope_kind else None
    a = om.new_seq(16)
    _, tok = a.prefill(emb, ids, pos)
    T, rope = a.len, a.rope_pos
    assert rope == (int(pos.max()) + 1 if rope_kind else T)

    def copy(rope_pos, drop_row=None):
        b = om.new_seq(16)
        for layer in range(cfg["n_layers"]):
            for sel in (0, 1):
                for head in range(cfg["n_kv_heads"]):
                    rows = a.read_kv(layer, sel, head, 0, T)
                    if drop_row is not None:
                        rows[drop_row] = 0.0
                    b.write_kv(layer, sel, head, 0, rows)
        b.set_len(T, rope_pos)
        return b

    b = copy(rope)
    for layer in range(cfg["n_layers"]):
        for head in range(cfg["n_kv_heads"]):
            assert np.array_equal(b.read_kv(layer, 0, head, 0, T), a.read_kv(layer, 0, head, 0, T))
    la, ha, ta = a.decode(tok)
    lb, hb, tb = b.decode(tok)
    assert np.array_equal(la, lb) and np.array_equal(ha, hb) and ta == tb
    assert b.len == a.len == T + 1 and b.rope_pos == a.rope_pos == rope + 1
    # the appended rows agree too
    for layer in range(cfg["n_layers"]):
        for sel in (0, 1):
            assert np.array_equal(a.read_kv(layer, sel, 0, T, 1), b.read_kv(layer, sel, 0, T, 1))
    lc, _, _ = copy(rope + 1).decode(tok)
    assert not np.array_equal(la, lc)
    ld, _, _ = copy(rope, drop_row=T // 2).decode(tok)
    assert not np.array_equal(la, ld)


def test_cache_copy_hooks_reject_out_of_range_rows():
    cfg = _cfg()
    om = O.Model(cfg, synth.make_weights(cfg))
    s = om.new_seq(4)
    rows = np.zeros((2, cfg["head_dim"]), np.float32)
    for bad in ((cfg["n_layers"], 0, 0, 0), (0, 2, 0, 0), (0, 0, cfg["n_kv_heads"], 0), (0, 0, 0, 3)):
        with pytest.raises(ValueError):
            s.write_kv(*bad, rows)
        with pytest.raises(ValueError):
            s.read_kv(*bad, 2)
    with pytest.raises(ValueError):
        s.set_len(5, 0)
    s.write_kv(0, 1, 1, 2, np.full((2, cfg["head_dim"]), 1.0 + 2.0 ** -12, np.float32))
    # write_kv stores R(.) of the rows: 1 + 2^-12 is a tie in binary16 and goes to even
    assert np.all(s.read_kv(0, 1, 1, 2, 2) == 1.0)
