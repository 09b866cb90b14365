"""The five workload shapes the decode path is tested and measured on.

Model shapes follow the two backbones of the paper's evaluation (§6.1
"Models"): a LLaVA-1.5-7B language model (Vicuna-7B: 32 layers, MHA with 32
KV heads) and a Qwen2.5-VL-7B language model (28 layers, GQA with 4 KV heads,
dynamic visual token counts).  The remaining hyper-parameters are those of the
public model cards (the Qwen-shaped model keeps its q/k/v biases); every
weight is random.  Each request stands in for one
image plus a short prompt and at most 128 generated tokens (§6.1
"Workload"); COCO images are replaced by seeded N(0, 1) vision rows.
"""
from __future__ import annotations

import copy

LLAVA7B = dict(n_layers=32, d_model=4096, n_heads=32, n_kv_heads=32, head_dim=128, ffn_dim=11008, vocab=32000,
               rope_theta=1e4, rms_eps=1e-5, rope_kind=0, mrope_section=(0, 0, 0), qkv_bias=0, dtype="f16")
QWEN25VL7B = dict(n_layers=28, d_model=3584, n_heads=28, n_kv_heads=4, head_dim=128, ffn_dim=18944,
                  vocab=152064, rope_theta=1e6, rms_eps=1e-6, rope_kind=1, mrope_section=(16, 24, 24),
                  qkv_bias=1, dtype="bf16")

CONFIGS = {
    # tiny fp32 decoder, batch 1: 576 vision rows + 32 text tokens, 16 greedy steps
    "tiny": dict(name="tiny", n_layers=2, d_model=256, n_heads=4, n_kv_heads=4, head_dim=64, ffn_dim=688,
                 vocab=1024, rope_theta=1e4, rms_eps=1e-5, rope_kind=0, mrope_section=(0, 0, 0), qkv_bias=0,
                 dtype="f32", batch=1, n_v=576, s_text=32, n_dec=16, seed=0),
    # LLaVA-1.5-7B-shaped fp16, batch 1: 576 vision rows + 64 text tokens, 128 steps
    "llava7b_b1": dict(LLAVA7B, name="llava7b_b1", batch=1, n_v=576, s_text=64, n_dec=128, seed=0),
    # same model, batch 32, text length uniform in [32, 256], 128 steps
    "llava7b_b32": dict(LLAVA7B, name="llava7b_b32", batch=32, n_v=576, s_text=(32, 256), n_dec=128, seed=0),
    # Qwen2.5-VL-7B-shaped bf16, batch 16, vision rows uniform in [256, 1280] + 128 text, 256 steps
    "qwen7b_b16": dict(QWEN25VL7B, name="qwen7b_b16", batch=16, n_v=(256, 1280), s_text=128, n_dec=256, seed=0),
    # one Qwen layer, bf16, batch 256, KV lengths uniform in [1024, 8192], 1000 appending steps
    "qwen_layer_b256": dict(QWEN25VL7B, name="qwen_layer_b256", n_layers=1, lm_head=False, batch=256,
                            kv_len=(1024, 8192), n_dec=1000, seed=0),
}

DTYPE_CODE = {"f32": 0, "f16": 1, "bf16": 2}
DTYPE_BYTES = {"f32": 4, "f16": 2, "bf16": 2}


def get(name: str, **overrides) -> dict:
    cfg = copy.deepcopy(CONFIGS[name])
    cfg.update(overrides)
    cfg.setdefault("lm_head", True)
    return cfg
