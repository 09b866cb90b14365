"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these compares the oracle with itself: each check is a value the paper
prints, a closed form, an invariant, a special case that reduces to a library
routine (numpy/torch conversions and ops, the transformers LLaMA and
Qwen2.5-VL text decoders), or brute force on tiny inputs.
"""
import json
import math
import os

import numpy as np
import pytest
import torch
from hypothesis import given, settings
from hypothesis import strategies as st

from oracle import oracle as O
from workload import configs, synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def mha_cfg(L, n_h, n_kv, d_h, d, dtype="f16"):
    return dict(n_layers=L, d_model=d, n_heads=n_h, n_kv_heads=n_kv, head_dim=d_h, ffn_dim=8, vocab=8,
                rope_theta=1e4, rms_eps=1e-5, rope_kind=0, mrope_section=(0, 0, 0), qkv_bias=0, dtype=dtype)


# ---------------------------------------------------------------------------
# Eq. 1, the embedding-size display and Theorem 1 (§4.1-4.2, Tables 2-3)
# ---------------------------------------------------------------------------

def test_transfer_sizes_match_paper_tables():
    with open(os.path.join(GOLDEN, "transfer_sizes.json")) as f:
        rows = json.load(f)["rows"]
    for row in rows:
        cfg = mha_cfg(row["L"], row["n_h"], row["n_kv"], row["d_h"], row["d"])
        kv, emb = O.transfer_bytes(cfg, row["n_v"], row["s_text"])
        if "kv_mib" in row:
            assert round(kv / 2**20) == row["kv_mib"], row["model"]
        if "emb_mib" in row:
            assert abs(emb / 2**20 - row["emb_mib"]) < 0.05 + 1e-9, row["model"]
        if "kv_bytes" in row:
            assert kv == row["kv_bytes"], row["model"]
        if "emb_bytes" in row:
            assert emb == row["emb_bytes"], row["model"]
        if "r_gqa" in row:
            assert round(kv / emb) == row["r_gqa"], row["model"]
        if "r_mha" in row:
            r_mha = 2 * row["L"] * (1 + row["s_text"] / row["n_v"])
            assert round(r_mha) == row["r_mha"], row["model"]


def test_worked_example_7b():
    # §4.1: 2 x 32 x 32 x 128 x 704 x 2 "~350 MB"; 576 x 4096 x 2 = 4.5 MB; ~78x
    cfg = dict(configs.LLAVA7B)
    kv, emb = O.transfer_bytes(cfg, 576, 128)
    assert kv == 2 * 32 * 32 * 128 * 704 * 2 == 369_098_752
    assert emb == 576 * 4096 * 2 == 4_718_592 == int(4.5 * 2**20)
    assert round(kv / emb) == 78
    # a prefill batch of 8 requests: "~2.8 GB" of KV (GiB)
    assert abs(8 * kv / 2**30 - 2.8) < 0.06
    # 128 images: "~576 MB" of embeddings
    assert 128 * emb == 576 * 2**20


def test_dynamic_resolution_embedding_size():
    # §4.2: N_v = 2048, d = 3584 -> "~14 MB"
    cfg = dict(configs.QWEN25VL7B)
    _, emb = O.transfer_bytes(cfg, 2048, 0)
    assert emb == 2048 * 3584 * 2 and round(emb / 2**20) == 14


@settings(max_examples=200, deadline=None)
@given(L=st.integers(1, 128), n_kv=st.integers(1, 64), g=st.integers(1, 8), d_h=st.sampled_from([32, 64, 128, 256]),
       n_v=st.integers(1, 4096), s_text=st.integers(0, 4096), dt=st.sampled_from(["f32", "f16", "bf16"]))
def test_theorem1_ratio_and_gqa_lower_bound(L, n_kv, g, d_h, n_v, s_text, dt):
    n_h = n_kv * g
    d = n_h * d_h
    cfg = mha_cfg(L, n_h, n_kv, d_h, d, dt)
    kv, emb = O.transfer_bytes(cfg, n_v, s_text)
    s_ctx = n_v + s_text
    # Eq. 2 as an exact integer identity: D_KV * N_v * d == D_emb * 2L n_kv d_h s_ctx
    assert kv * n_v * d == emb * 2 * L * n_kv * d_h * s_ctx
    # the byte width cancels (proof of Theorem 1)
    kv32, emb32 = O.transfer_bytes(dict(cfg, dtype="f32"), n_v, s_text)
    assert kv32 * emb == kv * emb32
    # GQA lower bound: R >= 2 L n_kv / n_h (s_text >= 0)
    assert kv * n_h >= 2 * L * n_kv * emb
    if g == 1:  # Eq. 3: R_MHA = 2L (1 + s_text / N_v), independent of d
        assert kv * n_v == emb * 2 * L * s_ctx


def test_transfer_bytes_rejects_bad_arguments():
    cfg = mha_cfg(2, 4, 4, 64, 256)
    with pytest.raises(ValueError):
        O.transfer_bytes(cfg, -1, 0)
    with pytest.raises(ValueError):
        O.transfer_bytes(dict(cfg, n_layers=0), 1, 0)


# ---------------------------------------------------------------------------
# storage rounding R(.) against library conversions
# ---------------------------------------------------------------------------

def _probe_values():
    rng = np.random.default_rng(0)
    v = np.concatenate([
        rng.standard_normal(20000).astype(np.float32),
        (rng.standard_normal(5000) * 1e-5).astype(np.float32),   # fp16 subnormal range
        (rng.standard_normal(5000) * 3e4).astype(np.float32),    # near fp16 overflow
        np.array([0.0, -0.0, 65504.0, 65519.99, 65520.0, 1e9, -1e9, 2**-24, 2**-25, 1.5 * 2**-25, 2**-26,
                  1.0 + 2**-11, 1.0 + 3 * 2**-11, 1.0 + 2**-8, 1.0 + 3 * 2**-8, np.inf, -np.inf], dtype=np.float32),
    ])
    return v


def test_round_f16_matches_numpy():
    v = _probe_values()
    want = v.astype(np.float16).view(np.uint16)
    got = np.array([O.f16_bits(x) for x in v], dtype=np.uint16)
    assert np.array_equal(got, want)


def test_round_bf16_matches_torch():
    v = _probe_values()
    want = torch.from_numpy(v).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    got = np.array([O.bf16_bits(x) for x in v], dtype=np.uint16)
    assert np.array_equal(got, want)


def test_round_is_identity_for_f32_and_nan_stays_nan():
    v = _probe_values()[:100]
    assert np.array_equal(O.round_to("f32", v), v)
    assert math.isnan(O.round_to("f16", [np.nan])[0]) and math.isnan(O.round_to("bf16", [np.nan])[0])


# ---------------------------------------------------------------------------
# RMSNorm, RoPE, attention, SiLU, argmax
# ---------------------------------------------------------------------------

def test_rmsnorm_closed_forms():
    d, eps = 64, 1e-5
    g = torch.ones(d, dtype=torch.float32)
    for c in (0.5, 3.0, -2.0):
        h = O.rmsnorm(np.full(d, c, np.float32), g, "f32", eps)
        assert np.allclose(h, c / math.sqrt(c * c + eps), rtol=1e-6)
    x = np.random.default_rng(1).standard_normal(d).astype(np.float32)
    gains = torch.from_numpy(np.random.default_rng(2).standard_normal(d).astype(np.float32))
    h1 = O.rmsnorm(x, gains, "f32", 0.0)
    h2 = O.rmsnorm(4.0 * x, gains, "f32", 0.0)  # scale invariance (exact power of two)
    assert np.allclose(h1, h2, rtol=1e-6, atol=0)
    ref = torch.nn.functional.rms_norm(torch.from_numpy(x).double(), (d,), gains.double(), eps).numpy()
    assert np.allclose(O.rmsnorm(x, gains, "f32", eps), ref, rtol=1e-6, atol=1e-7)


def _rope_cfg(d_h, kind=0, sec=(0, 0, 0), theta=1e4):
    return dict(n_layers=1, d_model=d_h, n_heads=1, n_kv_heads=1, head_dim=d_h, ffn_dim=8, vocab=8, rope_theta=theta,
                rms_eps=1e-5, rope_kind=kind, mrope_section=sec, qkv_bias=0, dtype="f32")


def test_rope_position_zero_is_identity_and_norm_preserved():
    cfg = _rope_cfg(128)
    v = np.random.default_rng(3).standard_normal(128).astype(np.float32)
    assert np.array_equal(O.rope_rotate(cfg, v, (0, 0, 0)), v)
    for p in (1, 17, 700, 8191):
        r = O.rope_rotate(cfg, v, (p, p, p))
        assert abs(np.linalg.norm(r) - np.linalg.norm(v)) < 1e-5 * np.linalg.norm(v)


def test_rope_pair_zero_turns_by_pos_radians():
    for p in (1, 5, 123):
        c, s = O.rope_cos_sin(1e4, 128, 0, p)
        assert c == np.float32(math.cos(p)) and s == np.float32(math.sin(p))
    c, s = O.rope_cos_sin(1e4, 128, 32, 1000)  # theta^(-1/2) = 1/100
    assert abs(c - math.cos(10.0)) < 1e-7 and abs(s - math.sin(10.0)) < 1e-7


def test_rope_scores_depend_only_on_relative_position():
    cfg = _rope_cfg(64)
    rng = np.random.default_rng(4)
    q, k = rng.standard_normal(64).astype(np.float32), rng.standard_normal(64).astype(np.float32)
    base = float(np.dot(O.rope_rotate(cfg, q, (9,) * 3), O.rope_rotate(cfg, k, (4,) * 3)))
    for shift in (1, 10, 100):
        m, n = 9 + shift, 4 + shift
        other = float(np.dot(O.rope_rotate(cfg, q, (m,) * 3), O.rope_rotate(cfg, k, (n,) * 3)))
        assert abs(other - base) < 2e-4 * (1 + abs(base))


def test_mrope_with_equal_ids_reduces_to_1d():
    rng = np.random.default_rng(5)
    v = rng.standard_normal(128).astype(np.float32)
    one = _rope_cfg(128, 0, theta=1e6)
    three = _rope_cfg(128, 1, (16, 24, 24), theta=1e6)
    for p in (0, 3, 999):
        assert np.array_equal(O.rope_rotate(one, v, (p, p, p)), O.rope_rotate(three, v, (p, p, p)))
    # each section follows its own id: rotate with (t, h, w) and compare every
    # pair with the 1-D rotation at that section's id
    t, h, w = 2, 30, 7
    r = O.rope_rotate(three, v, (t, h, w))
    for pair in range(64):
        p = t if pair < 16 else (h if pair < 40 else w)
        ref = O.rope_rotate(one, v, (p, p, p))
        assert r[pair] == ref[pair] and r[pair + 64] == ref[pair + 64]


def test_attention_single_key_returns_its_value():
    rng = np.random.default_rng(6)
    q, k, v = rng.standard_normal(8), rng.standard_normal((1, 8)), rng.standard_normal((1, 8))
    assert np.array_equal(O.attention(q, k, v), v[0].astype(np.float32))


def test_attention_identical_keys_return_mean_of_values():
    rng = np.random.default_rng(7)
    q = rng.standard_normal(16)
    k = np.tile(rng.standard_normal(16), (5, 1))
    v = rng.standard_normal((5, 16)).astype(np.float32)
    assert np.allclose(O.attention(q, k, v), v.astype(np.float64).mean(0), rtol=1e-6, atol=1e-7)


def test_attention_brute_force_and_library_sdpa():
    rng = np.random.default_rng(8)
    for n in range(1, 9):
        for d in (1, 2, 4, 8):
            q, k, v = (rng.standard_normal(s).astype(np.float32) for s in (d, (n, d), (n, d)))
            # brute force: enumerate exp(score) weights directly
            w = np.array([math.exp(float(np.dot(q.astype(np.float64), k[t].astype(np.float64))) / math.sqrt(d))
                          for t in range(n)])
            brute = (w[:, None] * v.astype(np.float64)).sum(0) / w.sum()
            got = O.attention(q, k, v)
            assert np.allclose(got, brute, rtol=1e-6, atol=1e-7)
            lib = torch.nn.functional.scaled_dot_product_attention(
                torch.from_numpy(q).double()[None, None, None], torch.from_numpy(k).double()[None, None],
                torch.from_numpy(v).double()[None, None])[0, 0, 0].numpy()
            assert np.allclose(got, lib, rtol=1e-6, atol=1e-7)
            perm = rng.permutation(n)
            assert np.allclose(O.attention(q, k[perm], v[perm]), got, rtol=1e-6, atol=1e-7)


def test_silu_and_argmax():
    assert O.silu(0.0) == 0.0
    z = torch.linspace(-20, 20, 401, dtype=torch.float32)
    ref = torch.nn.functional.silu(z.double()).numpy()
    got = np.array([O.silu(float(x)) for x in z])
    assert np.allclose(got, ref, rtol=1e-6, atol=1e-30)
    assert O.argmax([1.0, 3.0, 3.0, 2.0]) == 1  # lowest index on ties
    assert O.argmax([-1.0]) == 0
    assert O.argmax([0.0, float("nan")]) == -1


# ---------------------------------------------------------------------------
# whole model: library decoders, closed forms, consistency
# ---------------------------------------------------------------------------

def _tiny(**kw):
    base = dict(name="pin", n_layers=2, d_model=64, n_heads=4, n_kv_heads=4, head_dim=16, ffn_dim=96, vocab=97,
                rope_theta=1e4, rms_eps=1e-5, rope_kind=0, mrope_section=(0, 0, 0), qkv_bias=0, dtype="f32",
                lm_head=True, seed=11)
    base.update(kw)
    return base


def _hf_llama(cfg, W):
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
        sd.update({q + "self_attn.q_proj.weight": W[p + "wq"], q + "self_attn.k_proj.weight": W[p + "wk"],
                   q + "self_attn.v_proj.weight": W[p + "wv"], q + "self_attn.o_proj.weight": W[p + "wo"],
                   q + "mlp.gate_proj.weight": W[p + "w_gate"], q + "mlp.up_proj.weight": W[p + "w_up"],
                   q + "mlp.down_proj.weight": W[p + "w_down"], q + "input_layernorm.weight": W[p + "attn_norm"],
                   q + "post_attention_layernorm.weight": W[p + "mlp_norm"]})
    m.load_state_dict({k: v.double() for k, v in sd.items()})
    return m


def _rel(a, b):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    return float(np.max(np.abs(a - b)) / np.max(np.abs(b)))


def test_model_matches_transformers_llama_fp32():
    """With fp32 storage the oracle's decoder must reduce to the library LLaMA
    decoder run in fp64 (prefill from embeddings, then teacher-forced decode)."""
    cfg = _tiny(n_kv_heads=2)  # GQA, g = 2
    W = synth.make_weights(cfg)
    n_v, s_text = 7, 5
    emb = synth.vision_rows(cfg, 0, n_v)
    ids = synth.text_ids(cfg, 0, s_text)
    om = O.Model(cfg, W)
    seq = om.new_seq(n_v + s_text + 4)
    logits0, tok0 = seq.prefill(emb, ids)
    hf = _hf_llama(cfg, W)
    rows = [emb.double(), W["embed"].double()[ids.long()]]
    with torch.no_grad():
        ref = hf(inputs_embeds=torch.cat(rows)[None], use_cache=False).logits[0, -1].numpy()
    assert _rel(logits0, ref) < 1e-5
    toks = [tok0]
    for step in range(3):
        logits, _, tok = seq.decode(toks[-1])
        rows.append(W["embed"].double()[toks[-1]][None])
        with torch.no_grad():
            ref = hf(inputs_embeds=torch.cat(rows)[None], use_cache=False).logits[0, -1].numpy()
        assert _rel(logits, ref) < 1e-5
        assert tok == int(np.argmax(ref))
        toks.append(tok)


def test_model_matches_transformers_qwen25vl_text_mrope_bias():
    """M-RoPE (3 sections), GQA and q/k/v bias against the library Qwen2.5-VL
    text decoder in fp64."""
    from transformers.models.qwen2_5_vl.configuration_qwen2_5_vl import Qwen2_5_VLTextConfig
    from transformers.models.qwen2_5_vl.modeling_qwen2_5_vl import Qwen2_5_VLTextModel
    cfg = _tiny(n_heads=4, n_kv_heads=2, head_dim=16, rope_theta=1e6, rms_eps=1e-6, rope_kind=1,
                mrope_section=(2, 3, 3), qkv_bias=1)
    W = synth.make_weights(cfg)
    qc = Qwen2_5_VLTextConfig(vocab_size=cfg["vocab"], hidden_size=cfg["d_model"], intermediate_size=cfg["ffn_dim"],
                              num_hidden_layers=cfg["n_layers"], num_attention_heads=cfg["n_heads"],
                              num_key_value_heads=cfg["n_kv_heads"], rms_norm_eps=cfg["rms_eps"],
                              rope_parameters={"rope_type": "default", "rope_theta": cfg["rope_theta"],
                                               "mrope_section": list(cfg["mrope_section"])},
                              attn_implementation="eager", max_position_embeddings=4096,
                              bos_token_id=None, eos_token_id=None, pad_token_id=None)
    hf = Qwen2_5_VLTextModel(qc).double().eval()
    sd = {"embed_tokens.weight": W["embed"], "norm.weight": W["final_norm"]}
    for i in range(cfg["n_layers"]):
        p, q = f"layers.{i}.", f"layers.{i}."
        for a, b in (("wq", "self_attn.q_proj.weight"), ("wk", "self_attn.k_proj.weight"),
                     ("wv", "self_attn.v_proj.weight"), ("wo", "self_attn.o_proj.weight"),
                     ("bq", "self_attn.q_proj.bias"), ("bk", "self_attn.k_proj.bias"), ("bv", "self_attn.v_proj.bias"),
                     ("w_gate", "mlp.gate_proj.weight"), ("w_up", "mlp.up_proj.weight"),
                     ("w_down", "mlp.down_proj.weight"), ("attn_norm", "input_layernorm.weight"),
                     ("mlp_norm", "post_attention_layernorm.weight")):
            sd[q + b] = W[p + a]
    hf.load_state_dict({k: v.double() for k, v in sd.items()})
    n_v, s_text = 9, 4
    emb = synth.vision_rows(cfg, 0, n_v)
    ids = synth.text_ids(cfg, 0, s_text)
    pos = synth.mrope_positions(n_v, s_text)
    om = O.Model(cfg, W)
    seq = om.new_seq(n_v + s_text + 3)
    logits0, tok0 = seq.prefill(emb, ids, pos)
    assert seq.rope_pos == int(pos.max()) + 1
    rows = [emb.double(), W["embed"].double()[ids.long()]]
    lm = W["lm_head"].double()

    def ref_logits(positions):
        with torch.no_grad():
            h = hf(inputs_embeds=torch.cat(rows)[None], position_ids=positions[:, None, :].long(),
                   use_cache=False).last_hidden_state[0, -1]
        return (lm @ h).numpy()

    assert _rel(logits0, ref_logits(pos)) < 1e-5
    toks, positions = [tok0], pos
    for step in range(2):
        p = seq.rope_pos
        logits, _, tok = seq.decode(toks[-1])
        rows.append(W["embed"].double()[toks[-1]][None])
        positions = torch.cat([positions, torch.full((3, 1), p, dtype=torch.int32)], 1)
        ref = ref_logits(positions)
        assert _rel(logits, ref) < 1e-5
        toks.append(tok)


@pytest.mark.parametrize("dtype", ["f32", "f16", "bf16"])
def test_zero_blocks_reduce_to_embedding_head(dtype):
    """With W_o = W_down = 0 every layer leaves the residual unchanged, so the
    logits are W_lm . R(RMSNorm(E[t]) * g_f) (closed form)."""
    cfg = _tiny(dtype=dtype)
    W = synth.make_weights(cfg)
    for i in range(cfg["n_layers"]):
        W[f"layers.{i}.wo"] = torch.zeros_like(W[f"layers.{i}.wo"])
        W[f"layers.{i}.w_down"] = torch.zeros_like(W[f"layers.{i}.w_down"])
    om = O.Model(cfg, W)
    seq = om.new_seq(8)
    seq.prefill(None, [3, 5])
    logits, hidden, _ = seq.decode(42)
    e = W["embed"][42].double()
    assert np.array_equal(hidden, W["embed"][42].float().numpy())
    g = W["final_norm"].double()
    h = e / torch.sqrt((e * e).mean() + float(np.float32(cfg["rms_eps"]))) * g
    h = h.float().to({"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}[dtype]).double()
    ref = (W["lm_head"].double() @ h).numpy()
    assert _rel(logits, ref) < 1e-6


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_prefill_then_decode_equals_longer_prefill(dtype):
    """prefill(s + 1) last-row logits equal prefill(s) followed by decode(t_s)."""
    cfg = _tiny(dtype=dtype)
    W = synth.make_weights(cfg)
    om = O.Model(cfg, W)
    emb = synth.vision_rows(cfg, 0, 6)
    ids = synth.text_ids(cfg, 0, 4)
    a = om.new_seq(16)
    a.prefill(emb, ids[:3])
    la, _, _ = a.decode(int(ids[3]))
    b = om.new_seq(16)
    lb, _ = b.prefill(emb, ids)
    assert np.array_equal(la, lb)


def test_storage_rounding_stays_close_to_fp64_decoder():
    """fp16/bf16 storage only perturbs the fp64 library decoder by rounding."""
    for dtype, tol in (("f16", 5e-3), ("bf16", 4e-2)):
        cfg = _tiny(dtype=dtype)
        W = synth.make_weights(cfg)
        emb = synth.vision_rows(cfg, 0, 5)
        ids = synth.text_ids(cfg, 0, 3)
        logits, _ = O.Model(cfg, W).new_seq(10).prefill(emb, ids)
        hf = _hf_llama(cfg, {k: v.float() for k, v in W.items()})
        with torch.no_grad():
            ref = hf(inputs_embeds=torch.cat([emb.double(), W["embed"].double()[ids.long()]])[None],
                     use_cache=False).logits[0, -1].numpy()
        assert _rel(logits, ref) < tol, dtype


def test_state_and_capacity_errors():
    cfg = _tiny()
    om = O.Model(cfg, synth.make_weights(cfg))
    s = om.new_seq(4)
    with pytest.raises(ValueError):
        s.decode(1)                      # decode before prefill
    s.prefill(None, [1, 2, 3])
    with pytest.raises(ValueError):
        s.prefill(None, [1])             # prefill twice
    s.decode(1)
    with pytest.raises(ValueError):
        s.decode(1)                      # past capacity
    with pytest.raises(ValueError):
        om.new_seq(4).prefill(None, [cfg["vocab"]])  # token id out of range
